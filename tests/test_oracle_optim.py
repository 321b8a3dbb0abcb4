"""Pins of the oracle's Adam and of the GIST training loop built on it.

Adam (Kingma & Ba 2015, the optimizer of the paper's experiments):
* agrees with an independent implementation, ``torch.optim.Adam`` in fp64
  on the CPU, over many steps of random gradients;
* closed forms that bias correction fixes: the first step moves every weight
  by lr g / (|g| + eps) (a sign step), and under a constant gradient every
  step does the same, so k steps move by k lr g / (|g| + eps);
* with eps = 0 the update is invariant to a positive scaling of the gradients.

The loop (Algorithm 1 with Adam):
* m = 1 reproduces ordinary training of the full model (Section 2.1: one
  sub-GCN is the whole GCN), checked against a torch autograd + Adam loop:
  "carry" equals one optimizer kept across rounds, "reset" a fresh optimizer
  per round;
* with m > 1, entries that no sub-GCN owns keep their weights and zero
  moments, and the owned ones carry the moments their sub-GCN ended with.
"""

import numpy as np
import pytest
import torch

from gist_synth.graphs import erdos_renyi
from oracle import gist as G
from oracle import minibatch as MB
from oracle import optim as O
from oracle import partition as P


def test_adam_matches_torch():
    rng = np.random.default_rng(0)
    W0 = rng.standard_normal((7, 5))
    grads = [rng.standard_normal((7, 5)) * (0.1 + k) for k in range(25)]
    lr = 3e-3
    W, m, v = W0, np.zeros_like(W0), np.zeros_like(W0)
    for k, g in enumerate(grads, start=1):
        W, m, v = O.adam(W, g, m, v, k, lr)
    p = torch.nn.Parameter(torch.from_numpy(W0.copy()))
    opt = torch.optim.Adam([p], lr=lr, betas=(0.9, 0.999), eps=1e-8)
    for g in grads:
        p.grad = torch.from_numpy(g.copy())
        opt.step()
    want = p.detach().numpy()
    assert np.max(np.abs(W - want)) <= 1e-12 * np.max(np.abs(want))
    st = opt.state[p]
    # torch forms the moments with lerp (another rounding order): normwise
    for mine, theirs in ((m, st["exp_avg"].numpy()), (v, st["exp_avg_sq"].numpy())):
        assert np.max(np.abs(mine - theirs)) <= 1e-13 * np.max(np.abs(theirs))


def test_adam_first_step_is_a_sign_step():
    rng = np.random.default_rng(1)
    W = rng.standard_normal(100)
    g = rng.standard_normal(100) * np.logspace(-6, 3, 100)
    lr = 0.01
    W1, m1, v1 = O.adam(W, g, np.zeros(100), np.zeros(100), 1, lr)
    assert np.allclose(W - W1, lr * g / (np.abs(g) + O.EPS), rtol=1e-12, atol=0)
    assert np.allclose(m1, 0.1 * g) and np.allclose(v1, 0.001 * g * g)


def test_adam_constant_gradient_closed_form():
    rng = np.random.default_rng(2)
    W0 = rng.standard_normal(50)
    g = rng.standard_normal(50)
    lr = 1e-3
    W, m, v = W0, np.zeros(50), np.zeros(50)
    for k in range(1, 41):
        W, m, v = O.adam(W, g, m, v, k, lr)
    assert np.allclose(W0 - W, 40 * lr * g / (np.abs(g) + O.EPS), rtol=1e-10, atol=0)


def test_adam_scale_invariance():
    rng = np.random.default_rng(3)
    W0 = rng.standard_normal(30)
    gs = [rng.standard_normal(30) for _ in range(6)]
    out = []
    for c in (1.0, 1e4):
        W, m, v = W0, np.zeros(30), np.zeros(30)
        for k, g in enumerate(gs, start=1):
            W, m, v = O.adam(W, c * g, m, v, k, 0.05, eps=0.0)
        out.append(W)
    assert np.allclose(out[0], out[1], rtol=1e-12, atol=1e-14)


def test_adam_rejects_step_zero():
    with pytest.raises(ValueError):
        O.adam(np.zeros(2), np.ones(2), np.zeros(2), np.zeros(2), 0, 0.1)


# ---- the loop -------------------------------------------------------------

def _problem(seed=7, n=120, widths=(12, 16, 3)):
    g = erdos_renyi(n, 3 * n, seed)
    csr = MB.build(g, None, "gcn")
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((n, widths[0]))
    y = rng.integers(0, widths[-1], n).astype(np.int32)
    theta = [rng.standard_normal((widths[l], widths[l + 1])) * 0.3
             for l in range(len(widths) - 1)]
    return csr, X, y, theta


def _torch_train(csr, X, y, theta, steps_per_round, rounds, lr, fresh_each_round):
    """Plain full-model training with torch autograd + torch.optim.Adam (fp64)."""
    A = torch.from_numpy(MB.dense(csr))
    Xt = torch.from_numpy(X)
    yt = torch.from_numpy(y.astype(np.int64))
    Ws = [torch.nn.Parameter(torch.from_numpy(w.copy())) for w in theta]
    opt = None
    losses = []
    for t in range(rounds):
        if opt is None or fresh_each_round:
            opt = torch.optim.Adam(Ws, lr=lr)
        for _ in range(steps_per_round):
            H = Xt
            for l, W in enumerate(Ws):
                Z = A @ (H @ W)
                H = torch.relu(Z) if l < len(Ws) - 1 else Z
            loss = torch.nn.functional.cross_entropy(H, yt)
            opt.zero_grad()
            loss.backward()
            opt.step()
            losses.append(float(loss.detach()))
    return [w.detach().numpy() for w in Ws], losses


@pytest.mark.parametrize("policy", ["carry", "reset"])
def test_loop_m1_is_full_model_training(policy):
    csr, X, y, theta = _problem()
    rounds, zeta, lr = 3, 4, 0.01
    L = len(theta)
    parts = lambda t: [None] + [P.partition(theta[l].shape[0], 1, 100 * t + l)
                                for l in range(1, L)] + [None]
    got, Mg, Vg, losses = G.gist_train("gcn", theta, rounds, zeta, lr, parts,
                                       lambda t, i, z: (csr, X, y), policy=policy)
    want, wl = _torch_train(csr, X, y, theta, zeta, rounds, lr, policy == "reset")
    for a, b in zip(got, want):
        assert np.max(np.abs(a - b)) <= 1e-10 * np.max(np.abs(b))
    flat = [x for lt in losses for li in lt for x in li]
    assert np.allclose(flat, wl, rtol=1e-10, atol=0)
    assert flat[-1] < flat[0]


def test_loop_carry_moments_follow_ownership():
    csr, X, y, theta = _problem(widths=(12, 16, 8, 3))
    m, zeta, lr = 4, 2, 0.01
    L = len(theta)
    parts0 = [None] + [P.partition(theta[l].shape[0], m, 5 + l)
                       for l in range(1, L)] + [None]
    got, Mg, Vg, _ = G.gist_train("gcn", theta, 1, zeta, lr, lambda t: parts0,
                                  lambda t, i, z: (csr, X, y), policy="carry")
    # the hidden-to-hidden layer: owned entries are the diagonal blocks
    owned = np.zeros(theta[1].shape, bool)
    for i in range(m):
        r, c = G.slice_indices(parts0, L, i)[1]
        owned[np.ix_(r, c)] = True
    assert np.all(got[1][~owned] == theta[1][~owned])
    assert np.all(Mg[1][~owned] == 0) and np.all(Vg[1][~owned] == 0)
    # owned entries were trained (a dead ReLU unit may leave some at zero)
    assert np.mean(Vg[1][owned] > 0) > 0.5
    # every input-layer entry is owned by the sub-GCN of its column
    assert np.mean(Vg[0] > 0) > 0.5


def test_sgd_matches_torch():
    """``subTrain``'s plain SGD step (Section 2.2) against ``torch.optim.SGD``
    in fp64 over several steps with different learning rates and gradients:
    a wrong step size (2 lr, lr / n) or sign fails here."""
    from oracle import layers as Lr
    rng = np.random.default_rng(3)
    W0 = rng.standard_normal((6, 9))
    for lr in (0.5, 0.05, 1e-3):
        grads = [rng.standard_normal((6, 9)) * (1 + k) for k in range(6)]
        W = W0
        for g in grads:
            W = Lr.sgd(W, g, lr)
        p = torch.nn.Parameter(torch.from_numpy(W0.copy()))
        opt = torch.optim.SGD([p], lr=lr)
        for g in grads:
            opt.zero_grad()
            p.grad = torch.from_numpy(g.copy())
            opt.step()
        assert np.max(np.abs(W - p.detach().numpy())) <= 1e-12 * np.max(np.abs(W))
        # one step moves by exactly lr g: sign and size
        assert np.allclose(W0 - Lr.sgd(W0, grads[0], lr), lr * grads[0], rtol=0, atol=1e-15)


def test_grad_noise_hook_and_the_sensitivity_check():
    """``gist_train(grad_noise=...)`` leaves the run unchanged when absent and
    perturbs it when present; the element-wise Adam check the GPU training
    tests use (``tests/gpu_util.check_adam``) passes a run whose gradients
    carry rounding-sized noise and fails runs with a planted mistake: a step
    size off by 1%, or one element's update lost."""
    import sys
    import os
    sys.path.insert(0, os.path.dirname(__file__))
    from gpu_util import adam_noise, check_adam
    g = erdos_renyi(300, 900, 5)
    csr = MB.build(g, None, "gcn")
    rng = np.random.default_rng(11)
    widths, m = [24, 32, 16, 5], 2
    X = rng.standard_normal((g.n, widths[0]))
    y = rng.integers(0, widths[-1], g.n)
    theta = [rng.standard_normal((widths[l], widths[l + 1])) * 0.3 for l in range(3)]
    parts = lambda t: [None] + [P.partition(widths[l], m, 77 + 10 * t + l)
                                for l in (1, 2)] + [None]
    train = lambda noise, lr=0.01: G.gist_train("gcn", theta, 2, 2, lr, parts,
                                                lambda t, i, z: (csr, X, y), policy="reset",
                                                grad_noise=noise)[0]
    base = train(None)
    assert all(np.array_equal(a, b) for a, b in zip(base, train(None)))
    pert = [train(adam_noise(3e-6, s)) for s in (1, 2, 3)]
    assert any(not np.array_equal(a, b) for a, b in zip(base, pert[0]))
    change = lambda run: [run[l] - theta[l] for l in range(3)]
    want, ps = change(base), [change(q) for q in pert]
    # rounding-sized noise in the gradients: within the bound everywhere
    for l, got in enumerate(change(train(adam_noise(1e-6, 99)))):
        e_good, frac, ratio = check_adam(got, want[l], [q[l] for q in ps])
        assert e_good <= 1e-4 and ratio <= 1.0 and frac > 0.5
    # a 1% larger step size
    assert any(check_adam(got, want[l], [q[l] for q in ps])[2] > 1.0
               for l, got in enumerate(change(train(None, lr=0.0101))))
    # one well-conditioned element's update lost
    l = 1
    e = np.max([np.abs(q[l] - want[l]) for q in ps], axis=0)
    i = np.unravel_index(np.argmax(np.abs(want[l]) * (e <= 1e-5 * np.abs(want[l]).max())),
                         want[l].shape)
    got = want[l].copy()
    got[i] = 0.0
    e_good, _, ratio = check_adam(got, want[l], [q[l] for q in ps])
    assert e_good > 1e-4 and ratio > 1.0


@pytest.mark.parametrize("loop", ["sgd_round", "adam_train"])
def test_decision_overrides_in_the_loops(loop):
    """``masks`` and ``steps`` of ``gist_round`` / ``gist_train`` (test use:
    the GPU training tests run the oracle's backward through the GPU's own
    ReLU decisions).  Handing back the decisions the oracle itself took
    reproduces its run bit for bit; flipping one decision far from zero
    changes the trained weights; ``steps`` records every local step."""
    g = erdos_renyi(200, 700, 3)
    csr = MB.build(g, None, "gcn")
    rng = np.random.default_rng(5)
    widths, m, zeta = [10, 24, 12, 4], 2, 2
    X = rng.standard_normal((g.n, widths[0]))
    y = rng.integers(0, widths[-1], g.n)
    theta = [rng.standard_normal((widths[l], widths[l + 1])) * 0.4 for l in range(3)]
    parts = [None] + [P.partition(widths[l], m, 30 + l) for l in (1, 2)] + [None]

    def run(masks=None, steps=None):
        if loop == "sgd_round":
            mk = None if masks is None else (lambda i, z: masks[zeta * i + z])
            return G.gist_round("gcn", theta, parts, lambda i, z: (csr, X, y), 0.05, zeta,
                                masks=mk, steps=steps)[0]
        mk = None if masks is None else (lambda t, i, z: masks[zeta * i + z])
        return G.gist_train("gcn", theta, 1, zeta, 0.01, lambda t: parts,
                            lambda t, i, z: (csr, X, y), policy="carry", masks=mk,
                            steps=steps)[0]

    steps = []
    base = run(steps=steps)
    assert len(steps) == m * zeta
    own = [[st["recs"][l]["Z"] > 0 for l in range(2)] + [None] for st in steps]
    assert all(np.array_equal(a, b) for a, b in zip(base, run(masks=own)))
    # flip the decision of the largest pre-activation of sub-GCN 1's last step
    Z = steps[-1]["recs"][1]["Z"]
    i = np.unravel_index(np.argmax(np.abs(Z)), Z.shape)
    flipped = [[mk.copy() if mk is not None else None for mk in s] for s in own]
    flipped[-1][1][i] = not flipped[-1][1][i]
    assert any(not np.array_equal(a, b) for a, b in zip(base, run(masks=flipped)))
