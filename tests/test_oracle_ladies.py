"""Pins of the oracle's LADIES sampler and of GCN training on its per-layer
(rectangular) matrices (Section 5.4 and Appendix A.6: GIST with LADIES in
place of graph partitioning, vanilla GCN).

* closed forms: on a 3-node path with the middle node as the batch the
  distribution is p = (3/8, 1/4, 3/8) and the sampled row is
  (r, 1, r) / (1 + 2 r) with r = sqrt(2/3); on a complete graph every row of
  a sampled matrix is uniform over the sampled nodes;
* the importance q equals column sums of squares of the dense matrix (brute
  force), and the draws follow p (chi-square over many draws on a
  heavy-tailed graph, which a shifted index or a wrong prefix sum fails);
* invariants: V_L is the batch, V_{l+1} is inside V_l, |V_l| <= |V_{l+1}| + s,
  rows sum to one, a row's support is the sampled neighbourhood, entry
  ratios are (P_ij / p_j) / (P_ik / p_k), the stored transpose is the
  transpose; edge cases (no output node, s = 0, an isolated node);
* a sub-GCN step on the per-layer matrices equals torch autograd through
  dense rectangular matrices, and m = 1 GIST on LADIES batches with Adam is
  ordinary LADIES training of the full model.
"""

import numpy as np
import pytest
import torch

from gist_synth.graphs import Graph, chung_lu, erdos_renyi, sbm
from oracle import gist as G
from oracle import ladies as LD
from oracle import minibatch as MB
from oracle import partition as P


def _full(graph):
    return MB.build(graph, None, "gcn")


def _graph(n, edges):
    """A Graph from an explicit undirected edge list (one cluster)."""
    a = np.zeros((n, n), dtype=bool)
    for u, v in edges:
        a[u, v] = a[v, u] = True
    rowptr = np.concatenate([[0], np.cumsum(a.sum(1))]).astype(np.int64)
    col = np.concatenate([np.nonzero(a[i])[0] for i in range(n)] + [np.zeros(0, int)])
    return Graph(n, rowptr, col.astype(np.int32), np.array([0, n], np.int64),
                 np.arange(n, dtype=np.int32))


def test_path_closed_form():
    Pm = _full(_graph(3, [(0, 1), (1, 2)]))
    out = LD.sample(Pm, [1], 1, 64, seed=7)
    lay = out["layers"][0]
    assert np.allclose(lay["p"], [3 / 8, 1 / 4, 3 / 8], rtol=1e-6, atol=0)
    assert list(out["nodes"][0]) == [0, 1, 2]
    r = np.sqrt(2.0 / 3.0)
    want = np.array([[r, 1.0, r]]) / (1.0 + 2.0 * r)
    assert np.allclose(LD.dense(lay), want, rtol=1e-6, atol=0)


def test_complete_graph_rows_are_uniform():
    n = 7
    Pm = _full(_graph(n, [(i, j) for i in range(n) for j in range(i + 1, n)]))
    out = LD.sample(Pm, [0, 3], 2, 2, seed=99)
    for l, lay in enumerate(out["layers"]):
        assert np.allclose(lay["p"], 1.0 / n, rtol=1e-6, atol=0)
        D = LD.dense(lay)
        assert D.shape == (len(out["nodes"][l + 1]), len(out["nodes"][l]))
        assert np.allclose(D, 1.0 / D.shape[1], rtol=1e-6, atol=0)


def test_importance_is_column_norm_of_selected_rows():
    g = chung_lu(300, 2.5, 6.0, 5)
    Pm = _full(g)
    dense = MB.dense(Pm)
    rows = np.sort(np.random.default_rng(1).choice(300, 40, replace=False))
    q = LD.importance(Pm, rows)
    want = (dense[rows, :] ** 2).sum(axis=0)
    assert np.allclose(q, want, rtol=1e-14, atol=0)
    assert np.array_equal(q > 0, want > 0)


def test_draws_follow_the_distribution():
    g = chung_lu(400, 2.2, 8.0, 3)
    Pm = _full(g)
    rows = np.arange(0, 400, 9)
    q = LD.importance(Pm, rows)
    p = q / q.sum()
    k = 120_000
    d = np.asarray(LD.draw(q, k, P.SplitMix64(2024)))
    assert np.all(q[d] > 0)
    cnt = np.bincount(d, minlength=q.size)
    sel = p > 0
    # pool the sparse tail into one bin so every expected count is >= 5
    exp = k * p[sel]
    obs = cnt[sel].astype(np.float64)
    big = exp >= 5
    e2 = np.append(exp[big], exp[~big].sum())
    o2 = np.append(obs[big], obs[~big].sum())
    from scipy.stats import chi2
    stat = float(((o2 - e2) ** 2 / e2).sum())
    assert chi2.sf(stat, e2.size - 1) > 1e-6, stat
    # the distribution is far from uniform, so a shifted index would show
    assert p[sel].max() > 5 * p[sel].min()


@pytest.mark.parametrize("L,s,b", [(2, 64, 32), (3, 40, 17), (1, 200, 5)])
def test_invariants(L, s, b):
    g = sbm(1200, 12, 12.0, 0.8, 21)
    Pm = _full(g)
    dense = MB.dense(Pm)
    batch = np.sort(np.random.default_rng(L * 100 + s).choice(1200, b, replace=False))
    out = LD.sample(Pm, batch, L, s, seed=123 + L)
    V = out["nodes"]
    assert np.array_equal(V[L], batch)
    for l in range(L):
        lay = out["layers"][l]
        vin, vout = V[l], V[l + 1]
        assert np.all(np.diff(vin) > 0)
        assert set(vout.tolist()) <= set(vin.tolist())
        assert len(vin) <= len(vout) + s
        assert set(lay["draws"]) <= set(vin.tolist())
        assert set(vin.tolist()) == set(lay["draws"]) | set(vout.tolist())
        D = LD.dense(lay)
        assert D.shape == (len(vout), len(vin))
        assert np.allclose(D.sum(1), 1.0, rtol=0, atol=4e-7)
        sub = dense[np.ix_(vout, vin)]
        assert np.array_equal(D != 0, sub != 0)
        # ratios within a row follow P_ij / p_j
        p = lay["p"]
        for r in range(0, len(vout), max(1, len(vout) // 7)):
            nz = np.nonzero(D[r])[0]
            w = sub[r, nz] / p[vin[nz]]
            assert np.allclose(D[r, nz] / D[r, nz[0]], w / w[0], rtol=2e-6, atol=0)
        assert np.array_equal(LD.dense(lay, transpose=True), D.T)
    # reproducible; another seed draws differently
    again = LD.sample(Pm, batch, L, s, seed=123 + L)
    for a, c in zip(out["layers"], again["layers"]):
        assert a["draws"] == c["draws"]
        assert np.array_equal(a["val"].view(np.uint32), c["val"].view(np.uint32))
    other = LD.sample(Pm, batch, L, s, seed=124 + L)
    assert other["layers"][L - 1]["draws"] != out["layers"][L - 1]["draws"]


def test_edge_cases():
    g = _graph(5, [(0, 1), (1, 2)])          # nodes 3 and 4 are isolated
    Pm = _full(g)
    out = LD.sample(Pm, [], 2, 8, seed=1)
    assert all(v.size == 0 for v in out["nodes"])
    assert all(lay["nnz"] == 0 for lay in out["layers"])
    out = LD.sample(Pm, [4], 1, 8, seed=1)     # only node 4 has weight: every draw is 4
    assert out["layers"][0]["draws"] == [4] * 8
    assert list(out["nodes"][0]) == [4]
    assert np.array_equal(LD.dense(out["layers"][0]), [[1.0]])
    out = LD.sample(Pm, [0, 2], 2, 0, seed=1)  # s = 0: no draws, V_l = V_{l+1}
    for lay, v in zip(out["layers"], out["nodes"]):
        assert lay["draws"] == [] and list(v) == [0, 2]
        assert np.array_equal(LD.dense(lay), np.eye(2))   # 0 and 2 are not adjacent
    with pytest.raises(ValueError):
        LD.sample(Pm, [2, 1], 1, 4, seed=1)
    with pytest.raises(ValueError):
        LD.sample(Pm, [5], 1, 4, seed=1)


# ---- GCN on the per-layer matrices -----------------------------------------------

def _problem(seed=4, n=500, widths=(12, 20, 16, 5), b=24, s=48):
    g = erdos_renyi(n, 4 * n, seed)
    Pm = _full(g)
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((n, widths[0]))
    y = rng.integers(0, widths[-1], n).astype(np.int32)
    theta = [rng.standard_normal((widths[l], widths[l + 1])) * 0.3
             for l in range(len(widths) - 1)]
    L = len(widths) - 1

    def batch(key):
        r = np.random.default_rng(key)
        nodes = np.sort(r.choice(n, b, replace=False))
        out = LD.sample(Pm, nodes, L, s, seed=key)
        return out["layers"], X[out["nodes"][0]], y[out["nodes"][L]]
    return theta, batch


def _torch_run(layers, X, params):
    H = torch.from_numpy(X)
    L = len(params)
    for l, W in enumerate(params):
        A = torch.from_numpy(LD.dense(layers[l]))
        Z = (A @ H) @ W
        H = torch.relu(Z) if l < L - 1 else Z
    return H


def test_step_on_sampled_layers_matches_autograd():
    theta, batch = _problem()
    layers, X, y = batch(17)
    assert all(lay["n_in"] > lay["n"] for lay in layers)      # rectangular at every layer
    st = G.sub_gcn_step("gcn", layers, X, y, theta, 0.1)
    tp = [torch.tensor(w, requires_grad=True) for w in theta]
    out = _torch_run(layers, X, tp)
    assert out.shape[0] == len(y)
    loss = torch.nn.functional.cross_entropy(out, torch.from_numpy(y.astype(np.int64)))
    loss.backward()
    assert abs(float(loss.detach()) - st["loss"]) <= 1e-12 * abs(st["loss"])
    for l, w in enumerate(tp):
        want = w.grad.numpy()
        assert np.max(np.abs(st["grads"][l] - want)) <= 1e-10 * np.max(np.abs(want)), l


@pytest.mark.parametrize("policy", ["carry", "reset"])
def test_gist_m1_on_ladies_batches_is_ladies_training(policy):
    theta, batch = _problem(widths=(10, 16, 6), b=20, s=32)
    rounds, zeta, lr = 2, 3, 0.02
    L = len(theta)
    parts = lambda t: [None] + [P.partition(theta[l].shape[0], 1, 7 * t + l)
                                for l in range(1, L)] + [None]
    key = lambda t, i, z: 1000 * t + 10 * z + i
    got, _, _, losses = G.gist_train("gcn", theta, rounds, zeta, lr, parts,
                                     lambda t, i, z: batch(key(t, i, z)), policy=policy)
    ps = [torch.nn.Parameter(torch.from_numpy(w.copy())) for w in theta]
    opt, wl = None, []
    for t in range(rounds):
        if opt is None or policy == "reset":
            opt = torch.optim.Adam(ps, lr=lr)
        for z in range(zeta):
            layers, X, y = batch(key(t, 0, z))
            loss = torch.nn.functional.cross_entropy(_torch_run(layers, X, ps),
                                                     torch.from_numpy(y.astype(np.int64)))
            opt.zero_grad()
            loss.backward()
            opt.step()
            wl.append(float(loss.detach()))
    for a, b_ in zip(got, ps):
        b_ = b_.detach().numpy()
        assert np.max(np.abs(a - b_)) <= 1e-10 * np.max(np.abs(b_))
    flat = [x for lt in losses for li in lt for x in li]
    assert np.allclose(flat, wl, rtol=1e-10, atol=0)
