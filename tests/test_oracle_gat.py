"""Pins of the oracle's GAT layer (Velickovic et al. 2018, single head):

* central finite differences of every gradient (dW, da_src, da_dst, dH),
  with and without the ReLU, on a small graph;
* zero attention vectors make every score equal, so the layer reduces to the
  mean of P over N(i) u {i} -- checked against a dense (A + I) row mean built
  from the graph's edge list;
* with a LeakyReLU slope of 1 the score u_i + v_j is shifted by a per-row
  constant u_i, which the row softmax removes: the output does not depend
  on a_src and its gradient vanishes (a softmax over the wrong axis fails);
* attention rows are positive and sum to one; a node alone attends to itself.
"""

import numpy as np
import pytest

from gist_synth.graphs import erdos_renyi
from oracle import gat as GA
from oracle import minibatch as MB


def _setup(seed=0, n=14, s_in=5, s_out=4):
    g = erdos_renyi(n, 2 * n, seed)
    csr = MB.build(g, None, "gcn")   # pattern of A + I
    rng = np.random.default_rng(seed)
    H = rng.standard_normal((n, s_in))
    W = rng.standard_normal((s_in, s_out)) * 0.5
    a1 = rng.standard_normal(s_out)
    a2 = rng.standard_normal(s_out)
    R = rng.standard_normal((n, s_out))
    return g, csr, H, W, a1, a2, R


@pytest.mark.parametrize("act", [True, False])
def test_gat_finite_differences(act):
    g, csr, H, W, a1, a2, R = _setup()
    slope = 0.2
    f = GA.gat_forward(csr, H, W, a1, a2, act, slope)
    b = GA.gat_backward(csr, H, f, W, a1, a2, R, act, slope)

    def loss(H_, W_, a1_, a2_):
        return float(np.sum(GA.gat_forward(csr, H_, W_, a1_, a2_, act, slope)["H_out"] * R))

    eps = 1e-6
    for name, base, key in (("W", W, "dW"), ("a_src", a1, "da_src"), ("a_dst", a2, "da_dst"),
                            ("H", H, "dH")):
        num = np.zeros_like(base)
        it = np.nditer(base, flags=["multi_index"])
        for _ in it:
            idx = it.multi_index
            plus, minus = base.copy(), base.copy()
            plus[idx] += eps
            minus[idx] -= eps
            args_p = dict(H_=H, W_=W, a1_=a1, a2_=a2)
            args_m = dict(H_=H, W_=W, a1_=a1, a2_=a2)
            kw = {"W": "W_", "a_src": "a1_", "a_dst": "a2_", "H": "H_"}[name]
            args_p[kw], args_m[kw] = plus, minus
            num[idx] = (loss(**args_p) - loss(**args_m)) / (2 * eps)
        assert np.max(np.abs(num - b[key])) <= 1e-6 * max(1.0, np.max(np.abs(num))), name


def test_gat_zero_attention_is_mean_over_self_and_neighbours():
    g, csr, H, W, a1, a2, R = _setup(seed=1)
    f = GA.gat_forward(csr, H, W, np.zeros_like(a1), np.zeros_like(a2), False, 0.2)
    # dense A + I from the graph's own edge list
    n = g.n
    A = np.eye(n)
    rp, col = np.asarray(g.rowptr), np.asarray(g.col)
    for i in range(n):
        A[i, col[rp[i]:rp[i + 1]]] = 1.0
    mean = (A / A.sum(1, keepdims=True)) @ (H @ W)
    assert np.allclose(f["Z"], mean, rtol=1e-12, atol=1e-12)


def test_gat_slope_one_ignores_a_src():
    g, csr, H, W, a1, a2, R = _setup(seed=2)
    f1 = GA.gat_forward(csr, H, W, a1, a2, True, 1.0)
    f2 = GA.gat_forward(csr, H, W, 3.0 * a1 - 1.0, a2, True, 1.0)
    assert np.allclose(f1["H_out"], f2["H_out"], rtol=1e-12, atol=1e-12)
    b = GA.gat_backward(csr, H, f1, W, a1, a2, R, True, 1.0)
    assert np.max(np.abs(b["da_src"])) <= 1e-12 * np.max(np.abs(b["da_dst"]))


def test_gat_attention_rows_are_distributions():
    g, csr, H, W, a1, a2, R = _setup(seed=3)
    f = GA.gat_forward(csr, H, W, a1, a2, True, 0.2)
    rp = np.asarray(csr["rowptr"])
    sums = np.add.reduceat(f["alpha"], rp[:-1])
    assert np.all(f["alpha"] > 0) and np.allclose(sums, 1.0, rtol=0, atol=1e-14)


def test_gat_single_node_attends_to_itself():
    csr = dict(n=1, nnz=1, rowptr=np.array([0, 1]), col=np.array([0], np.int32),
               val=np.array([1.0], np.float32))
    rng = np.random.default_rng(4)
    H, W = rng.standard_normal((1, 3)), rng.standard_normal((3, 2))
    f = GA.gat_forward(csr, H, W, rng.standard_normal(2), rng.standard_normal(2), False, 0.2)
    assert np.allclose(f["alpha"], [1.0]) and np.allclose(f["Z"], H @ W)


def test_gat_decision_overrides():
    """``pos`` = the oracle's own LeakyReLU sides and ``mask`` = its own ReLU
    decisions reproduce the backward bit for bit; with slope 1 the LeakyReLU
    is the identity, so any choice of sides gives the same gradients; with
    slope 0.2 flipping one entry's side scales that entry's gradient by 0.2
    or 1 / 0.2 and changes du of its row and dv of its column by the
    difference, and nothing else of du, dv."""
    g, csr, H, W, a1, a2, R = _setup(seed=4)
    for slope in (1.0, 0.2):
        f = GA.gat_forward(csr, H, W, a1, a2, True, slope)
        base = GA.gat_backward(csr, H, f, W, a1, a2, R, True, slope)
        same = GA.gat_backward(csr, H, f, W, a1, a2, R, True, slope, mask=f["Z"] > 0,
                               pos=f["pre"] > 0)
        for k in base:
            assert np.array_equal(base[k], same[k])
        pos = f["pre"] > 0
        rng = np.random.default_rng(1)
        flips = rng.random(pos.shape) < 0.3
        other = GA.gat_backward(csr, H, f, W, a1, a2, R, True, slope, pos=pos ^ flips)
        if slope == 1.0:
            for k in ("dW", "da_src", "da_dst", "dH"):
                assert np.array_equal(other[k], base[k])
    # slope 0.2, one flip: entry e of row i, column j
    rp = np.asarray(csr["rowptr"])
    i = 5
    e = next(k for k in range(int(rp[i]), int(rp[i + 1])) if int(csr["col"][k]) != i)
    j = int(csr["col"][e])
    pos1 = pos.copy()
    pos1[e] = not pos1[e]
    one = GA.gat_backward(csr, H, f, W, a1, a2, R, True, 0.2, pos=pos1)
    # only the entry's own gradient changes, by the ratio of the two slopes
    ratio = 0.2 if pos[e] else 1.0 / 0.2
    assert one["dpre"][e] == pytest.approx(ratio * base["dpre"][e], rel=1e-12)
    others = np.arange(len(pos)) != e
    assert np.array_equal(one["dpre"][others], base["dpre"][others])
    d_u, d_v = one["du"] - base["du"], one["dv"] - base["dv"]
    step = one["dpre"][e] - base["dpre"][e]
    assert d_u[i] == pytest.approx(step, rel=1e-9) and d_v[j] == pytest.approx(step, rel=1e-9)
    assert np.all(d_u[np.arange(len(d_u)) != i] == 0.0)
    assert np.all(d_v[np.arange(len(d_v)) != j] == 0.0)
