"""Pins of the oracle's step and round (Algorithm 1; Sections 2.1-2.2; Appendix C).

* m = 1: the single sub-GCN is the full GCN;
* two layers with unpartitioned input and output: the full model's logits
  are the sum of the m sub-GCN logits (each hidden unit lives in exactly one
  block, and the activation is elementwise), for GCN and SAGE-mean;
* after ``subAgg`` the two-layer full model equals the sum of the trained
  sub-GCNs; entries outside every block are untouched; a skipped worker
  leaves its block at the old values;
* Appendix C's procedure: the additive form theta + sum_j (theta_j,zeta -
  theta_j,0) equals replacement; the aggregated 1/m-scaled model satisfies
  the global error decomposition lemma.
"""

import numpy as np
import pytest

from gist_synth.graphs import erdos_renyi, sbm
from oracle import gist as G
from oracle import layers as Lr
from oracle import minibatch as MB
from oracle import partition as P


def rand_theta(kind, widths, rng):
    th = []
    for l in range(len(widths) - 1):
        if kind == "gcn":
            th.append(rng.standard_normal((widths[l], widths[l + 1])) * 0.5)
        else:
            th.append((rng.standard_normal((widths[l], widths[l + 1])) * 0.5,
                       rng.standard_normal((widths[l], widths[l + 1])) * 0.5))
    return th


def partitions_for(widths, m, seed):
    L = len(widths) - 1
    parts = [None] * (L + 1)
    for l in range(1, L):
        parts[l] = P.partition(widths[l], m, seed + l)
    return parts


@pytest.fixture(scope="module")
def setup():
    g = erdos_renyi(40, 80, seed=4)
    rng = np.random.default_rng(12)
    X = rng.standard_normal((40, 9))
    y = rng.integers(0, 5, 40)
    return g, X, y, rng


@pytest.mark.parametrize("kind", ["gcn", "sage"])
def test_m1_is_full_model(setup, kind):
    g, X, y, rng = setup
    csr = MB.build(g, None, "gcn" if kind == "gcn" else "sage")
    widths = [9, 12, 10, 5]
    th = rand_theta(kind, widths, rng)
    parts = partitions_for(widths, 1, 3)
    sub = G.gather_params(kind, th, G.slice_indices(parts, 3, 0))
    a = G.sub_gcn_step(kind, csr, X, y, sub, 0.1)
    b = G.sub_gcn_step(kind, csr, X, y, th, 0.1)
    assert a["loss"] == b["loss"]
    assert np.array_equal(a["H"][-1], b["H"][-1])


@pytest.mark.parametrize("kind", ["gcn", "sage"])
@pytest.mark.parametrize("m", [2, 4])
def test_two_layer_sum_identity(setup, kind, m):
    g, X, y, rng = setup
    csr = MB.build(g, None, "gcn" if kind == "gcn" else "sage")
    widths = [9, 16, 5]
    th = rand_theta(kind, widths, rng)
    parts = partitions_for(widths, m, 40)
    full, _ = G.forward(kind, csr, X, th)
    total = np.zeros_like(full[-1])
    for i in range(m):
        sub = G.gather_params(kind, th, G.slice_indices(parts, 2, i))
        H, _ = G.forward(kind, csr, X, sub)
        total += H[-1]
    assert np.max(np.abs(total - full[-1])) <= 1e-13 * np.max(np.abs(full[-1]))


@pytest.mark.parametrize("kind", ["gcn", "sage"])
def test_round_aggregate_equals_sum_of_trained(setup, kind):
    g, X, y, rng = setup
    norm = "gcn" if kind == "gcn" else "sage"
    csr = MB.build(g, None, norm)
    widths = [9, 16, 5]
    m = 4
    th = rand_theta(kind, widths, rng)
    parts = partitions_for(widths, m, 70)
    new, trained, losses = G.gist_round(kind, th, parts, lambda i, z: (csr, X, y),
                                        lr=0.05, zeta=3)
    full, _ = G.forward(kind, csr, X, new)
    total = sum(G.forward(kind, csr, X, p)[0][-1] for p in trained)
    assert np.max(np.abs(total - full[-1])) <= 1e-12 * np.max(np.abs(full[-1]))
    # local steps decrease each sub-GCN's training loss on this tiny problem
    assert all(l[-1] < l[0] for l in losses)


def test_round_on_clusters_untouched_entries_and_skipped_worker():
    g = sbm(300, 10, 12.0, 0.9, seed=8)
    rng = np.random.default_rng(3)
    X = rng.standard_normal((300, 6))
    y = rng.integers(0, 4, 300)
    kind, widths, m = "sage", [6, 8, 8, 4], 2
    th = rand_theta(kind, widths, rng)
    parts = partitions_for(widths, m, 9)

    def batches(i, z):
        csr = MB.build(g, [i, 5 + z], "sage")
        nm = csr["node_map"]
        return csr, X[nm], y[nm]

    new, trained, _ = G.gist_round(kind, th, parts, batches, lr=0.1, zeta=2)
    # hidden layer 1: entries with row and column in different blocks stay
    for part in range(2):
        b0 = P.blocks_of(*parts[1])
        b1 = P.blocks_of(*parts[2])
        keep = np.ones((8, 8), dtype=bool)
        for i in range(m):
            keep[np.ix_(b0[i], b1[i])] = False
        assert np.array_equal(new[1][part][keep], th[1][part][keep])
        assert not np.array_equal(new[1][part][~keep], th[1][part][~keep])
    # skip sub-GCN 1's subAgg: its blocks keep the old values
    partial = G.scatter_params(kind, th, G.slice_indices(parts, 3, 0), trained[0])
    sl1 = G.slice_indices(parts, 3, 1)
    for l, (r, c) in enumerate(sl1):
        for part in range(2):
            assert np.array_equal(Lr.gather_slice(partial[l][part], r, c),
                                  Lr.gather_slice(th[l][part], r, c))


def test_theory_procedure_additive_equals_replace_and_error_decomposition():
    """Appendix C.1 procedure and the global error decomposition lemma."""
    n, d, d1, m, zeta, eta = 8, 3, 16, 4, 3, 0.05
    g = erdos_renyi(n, 12, seed=13)
    csr = MB.build(g, None, "theory")
    rng = np.random.default_rng(14)
    X = rng.standard_normal((n, d)) * 0.3
    Theta = rng.standard_normal((d, d1))
    a = rng.choice([-1.0, 1.0], size=d1)
    y = rng.standard_normal(n)
    idx, offs = P.partition(d1, m, 5)
    blocks = P.blocks_of(idx, offs)

    def sub_out(Th, Dj):
        W1 = (a[Dj] / np.sqrt(d1))[:, None]
        f0 = Lr.gcn_forward(csr, X, Th[:, Dj], True)
        return Lr.gcn_forward(csr, f0["H_out"], W1, False)["H_out"][:, 0]

    def step(Th, Dj):
        W0 = Th[:, Dj]
        W1 = (a[Dj] / np.sqrt(d1))[:, None]
        f0 = Lr.gcn_forward(csr, X, W0, True)
        f1 = Lr.gcn_forward(csr, f0["H_out"], W1, False)
        r = f1["H_out"] - y[:, None]       # gradient of the halved squared loss
        b1 = Lr.gcn_backward(csr, f0["H_out"], f1, W1, r, False)
        b0 = Lr.gcn_backward(csr, X, f0, W0, b1["dH"], True, need_dH=False)
        out = Th.copy()
        out[:, Dj] = Lr.sgd(W0, b0["dW"], eta)
        return out

    trained = []
    for Dj in blocks:
        Th = Theta.copy()
        for _ in range(zeta):
            Th = step(Th, Dj)
        trained.append(Th)
    additive = Theta + sum(T - Theta for T in trained)
    replaced = Theta.copy()
    for Dj, T in zip(blocks, trained):
        replaced = Lr.subagg(replaced, None, Dj, T[:, Dj])
    assert np.max(np.abs(additive - replaced)) < 1e-14
    # 1/m-scaled full model after aggregation is the mean of the sub-GCN outputs
    yh = [sub_out(T, Dj) for T, Dj in zip(trained, blocks)]
    full = sub_out(replaced, list(range(d1))) / m
    assert np.allclose(full, np.mean(yh, axis=0), rtol=0, atol=1e-13)
    lhs = np.sum((y - full) ** 2)
    rhs = (np.mean([np.sum((y - v) ** 2) for v in yh])
           - sum(np.sum((yh[j] - yh[jj]) ** 2) for j in range(m) for jj in range(j))
           / m ** 2)
    assert lhs == pytest.approx(rhs, rel=1e-12)
