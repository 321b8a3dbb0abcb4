"""Pins of the oracle's GAT models under GIST (sub-GCN step, subAgg, loop).

* the sub-GCN step's gradients of a 3-layer GAT model equal torch autograd
  through a dense formulation of the same model (attention as a masked row
  softmax of a full n x n score matrix), which shares nothing with the
  oracle's sparse forward and hand-written backward;
* m = 1 GIST training with Adam is ordinary training of the full GAT model
  (Section 2.1), against torch autograd + torch.optim.Adam, both moment
  policies;
* subAgg: every sub-GCN re-gathers exactly its trained slices (matrices and
  hidden-layer attention vectors); the output layer's shared attention
  vectors are the mean of the m trained copies, i.e. the deviations of the
  copies from the aggregate sum to zero and the aggregate lies between the
  smallest and largest copy; a round with lr = 0 leaves Theta bitwise as it
  was (gather, identity training, replacement, mean of equal copies).
"""

import numpy as np
import pytest
import torch

from gist_synth.graphs import erdos_renyi
from oracle import gist as G
from oracle import minibatch as MB
from oracle import partition as P


def _problem(seed=11, n=90, widths=(10, 16, 12, 4)):
    g = erdos_renyi(n, 3 * n, seed)
    csr = MB.build(g, None, "gcn")      # pattern of A + I
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((n, widths[0]))
    y = rng.integers(0, widths[-1], n).astype(np.int32)
    theta = [(rng.standard_normal((widths[l], widths[l + 1])) * 0.4,
              rng.standard_normal(widths[l + 1]) * 0.3,
              rng.standard_normal(widths[l + 1]) * 0.3) for l in range(len(widths) - 1)]
    return csr, X, y, theta


def _torch_model(csr):
    mask = torch.from_numpy(MB.dense(csr) != 0)

    def run(X, params):
        H = X
        L = len(params)
        for l, (W, a1, a2) in enumerate(params):
            Pm = H @ W
            e = torch.nn.functional.leaky_relu((Pm @ a1)[:, None] + (Pm @ a2)[None, :],
                                               G.GAT_SLOPE)
            alpha = torch.softmax(e.masked_fill(~mask, float("-inf")), dim=1)
            Z = alpha @ Pm
            H = torch.relu(Z) if l < L - 1 else Z
        return H
    return run


def test_gat_step_gradients_match_autograd():
    csr, X, y, theta = _problem()
    st = G.sub_gcn_step("gat", csr, X, y, theta, 0.1)
    run = _torch_model(csr)
    tp = [tuple(torch.tensor(x, requires_grad=True) for x in layer) for layer in theta]
    out = run(torch.from_numpy(X), tp)
    loss = torch.nn.functional.cross_entropy(out, torch.from_numpy(y.astype(np.int64)))
    loss.backward()
    assert abs(float(loss.detach()) - st["loss"]) <= 1e-12 * abs(st["loss"])
    for l in range(len(theta)):
        for k in range(3):
            want = tp[l][k].grad.numpy()
            got = st["grads"][l][k]
            assert np.max(np.abs(got - want)) <= 1e-10 * np.max(np.abs(want)), (l, k)


def _torch_train(csr, X, y, theta, zeta, rounds, lr, fresh_each_round):
    run = _torch_model(csr)
    ps = [torch.nn.Parameter(torch.from_numpy(x.copy())) for layer in theta for x in layer]
    yt = torch.from_numpy(y.astype(np.int64))
    opt, losses = None, []
    for _ in range(rounds):
        if opt is None or fresh_each_round:
            opt = torch.optim.Adam(ps, lr=lr)
        for _ in range(zeta):
            params = [tuple(ps[3 * l:3 * l + 3]) for l in range(len(theta))]
            loss = torch.nn.functional.cross_entropy(run(torch.from_numpy(X), params), yt)
            opt.zero_grad()
            loss.backward()
            opt.step()
            losses.append(float(loss.detach()))
    return [tuple(p.detach().numpy() for p in ps[3 * l:3 * l + 3]) for l in range(len(theta))], losses


@pytest.mark.parametrize("policy", ["carry", "reset"])
def test_gat_loop_m1_is_full_model_training(policy):
    csr, X, y, theta = _problem()
    rounds, zeta, lr = 2, 3, 0.01
    L = len(theta)
    parts = lambda t: [None] + [P.partition(theta[l][0].shape[0], 1, 50 * t + l)
                                for l in range(1, L)] + [None]
    got, _, _, losses = G.gist_train("gat", theta, rounds, zeta, lr, parts,
                                     lambda t, i, z: (csr, X, y), policy=policy)
    want, wl = _torch_train(csr, X, y, theta, zeta, rounds, lr, policy == "reset")
    for gl, wl_ in zip(got, want):
        for a, b in zip(gl, wl_):
            assert np.max(np.abs(a - b)) <= 1e-10 * np.max(np.abs(b))
    flat = [x for lt in losses for li in lt for x in li]
    assert np.allclose(flat, wl, rtol=1e-10, atol=0)


def _round(lr, m=4, seed=3):
    csr, X, y, theta = _problem()
    L = len(theta)
    parts = [None] + [P.partition(theta[l][0].shape[0], m, seed + l) for l in range(1, L)] + [None]
    new, trained, _ = G.gist_round("gat", theta, parts, lambda i, z: (csr, X, y), lr, zeta=2)
    return theta, new, trained, parts


def test_gat_subagg_replaces_slices_and_averages_shared_vectors():
    theta, new, trained, parts = _round(0.05)
    L, m = len(theta), len(trained)
    for i in range(m):
        sl = G.slice_indices(parts, L, i)
        again = G.gather_params("gat", new, sl)
        for l in range(L):
            last = l == L - 1
            for k in range(3):
                if last and k > 0:
                    continue        # shared: checked below
                assert np.array_equal(again[l][k], trained[i][l][k]), (i, l, k)
    for k in (1, 2):
        copies = np.stack([trained[i][L - 1][k] for i in range(m)])
        agg = new[L - 1][k]
        assert not np.allclose(copies[0], copies[1])        # the copies did diverge
        dev = np.sum(copies - agg[None, :], axis=0)
        assert np.max(np.abs(dev)) <= 1e-14 * np.max(np.abs(copies))
        assert np.all(agg >= copies.min(0)) and np.all(agg <= copies.max(0))


def test_gat_round_without_learning_keeps_theta():
    theta, new, _, _ = _round(0.0)
    for a, b in zip(theta, new):
        for x, y_ in zip(a, b):
            assert np.array_equal(np.asarray(x, np.float64), y_)
