"""Pins of the oracle's layer forward/backward and loss.

* central finite differences of the forward give the backward;
* special graphs reduce the layer to plain dense products: no edges
  (GCN: Abar = I), the complete graph (every aggregated row is the mean),
  a star (SAGE-mean: centre gets the leaves' mean, leaves get the centre);
* the one-hidden-layer theory model's closed-form gradient (Appendix C.1,
  with the squared loss halved so the printed gradient has no factor 2) is
  reproduced by the generic layer backward;
* softmax cross-entropy: uniform logits give log C.
"""

import numpy as np
import pytest

from gist_synth.graphs import Graph, _csr_from_undirected, erdos_renyi
from oracle import layers as Lr
from oracle import minibatch as MB
from oracle import partition as P


def graph_from_edges(n, edges):
    rowptr, col = _csr_from_undirected(n, [a for a, b in edges], [b for a, b in edges])
    return Graph(n, rowptr, col, np.array([0, n], dtype=np.int64),
                 np.arange(n, dtype=np.int32))


def fd_grad(f, x, eps=1e-6):
    g = np.zeros_like(x)
    it = np.nditer(x, flags=["multi_index"])
    for _ in it:
        i = it.multi_index
        old = x[i]
        x[i] = old + eps
        fp = f()
        x[i] = old - eps
        fm = f()
        x[i] = old
        g[i] = (fp - fm) / (2 * eps)
    return g


def rel(a, b):
    return np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-30)


@pytest.fixture(scope="module")
def tiny():
    g = erdos_renyi(7, 9, seed=2)
    rng = np.random.default_rng(0)
    return g, rng


@pytest.mark.parametrize("act", [True, False])
def test_gcn_backward_matches_finite_differences(tiny, act):
    g, rng = tiny
    csr = MB.build(g, None, "gcn")
    H = rng.standard_normal((7, 5))
    W = rng.standard_normal((5, 4))
    R = rng.standard_normal((7, 4))

    def f():
        return float((Lr.gcn_forward(csr, H, W, act)["H_out"] * R).sum())

    fwd = Lr.gcn_forward(csr, H, W, act)
    assert np.min(np.abs(fwd["Z"])) > 1e-4  # away from the ReLU kink
    b = Lr.gcn_backward(csr, H, fwd, W, R, act)
    assert rel(b["dW"], fd_grad(f, W)) < 1e-6
    assert rel(b["dH"], fd_grad(f, H)) < 1e-6


@pytest.mark.parametrize("act", [True, False])
def test_sage_backward_matches_finite_differences(tiny, act):
    g, rng = tiny
    csr = MB.build(g, None, "sage")
    H = rng.standard_normal((7, 5))
    Ws = rng.standard_normal((5, 3))
    Wn = rng.standard_normal((5, 3))
    R = rng.standard_normal((7, 3))

    def f():
        return float((Lr.sage_forward(csr, H, Ws, Wn, act)["H_out"] * R).sum())

    fwd = Lr.sage_forward(csr, H, Ws, Wn, act)
    assert np.min(np.abs(fwd["Z"])) > 1e-4
    b = Lr.sage_backward(csr, H, fwd, Ws, Wn, R, act)
    assert rel(b["dW_self"], fd_grad(f, Ws)) < 1e-6
    assert rel(b["dW_neigh"], fd_grad(f, Wn)) < 1e-6
    assert rel(b["dH"], fd_grad(f, H)) < 1e-6


def test_softmax_xent_finite_differences_and_uniform():
    rng = np.random.default_rng(1)
    Z = rng.standard_normal((6, 5))
    y = rng.integers(0, 5, 6)
    loss, dZ = Lr.softmax_xent(Z, y)
    assert rel(dZ, fd_grad(lambda: Lr.softmax_xent(Z, y)[0], Z)) < 1e-6
    assert np.allclose(dZ.sum(axis=1), 0.0, atol=1e-15)
    l0, _ = Lr.softmax_xent(np.full((4, 7), 3.25), [0, 1, 6, 3])
    assert l0 == pytest.approx(np.log(7.0), abs=1e-14)
    with pytest.raises(ValueError):
        Lr.softmax_xent(Z, [5, 0, 0, 0, 0, 0])


def test_edgeless_gcn_is_dense_product():
    g = graph_from_edges(5, [])
    csr = MB.build(g, None, "gcn")
    rng = np.random.default_rng(3)
    H, W = rng.standard_normal((5, 4)), rng.standard_normal((4, 3))
    out = Lr.gcn_forward(csr, H, W, True)
    assert np.array_equal(out["H_out"], np.maximum(H @ W, 0.0))


def test_complete_graph_aggregates_the_mean():
    n = 6
    g = graph_from_edges(n, [(i, j) for i in range(n) for j in range(i + 1, n)])
    csr = MB.build(g, None, "gcn")
    H = np.random.default_rng(4).standard_normal((n, 3))
    AH = Lr.aggregate(csr, H)
    assert np.allclose(AH, np.tile(H.mean(axis=0), (n, 1)), rtol=1e-6)


def test_sage_star_and_edgeless():
    g = graph_from_edges(5, [(0, k) for k in range(1, 5)])
    csr = MB.build(g, None, "sage")
    rng = np.random.default_rng(5)
    H = rng.standard_normal((5, 3))
    AH = Lr.aggregate(csr, H)
    assert np.allclose(AH[0], H[1:].mean(axis=0), rtol=1e-6)
    for k in range(1, 5):
        assert np.array_equal(AH[k], H[0])
    ge = graph_from_edges(4, [])
    ce = MB.build(ge, None, "sage")
    Ws, Wn = rng.standard_normal((3, 2)), rng.standard_normal((3, 2))
    X = rng.standard_normal((4, 3))
    out = Lr.sage_forward(ce, X, Ws, Wn, False)
    assert np.array_equal(out["AH"], np.zeros((4, 3)))
    assert np.array_equal(out["Z"], X @ Ws)


def test_association_orders_agree(tiny):
    g, rng = tiny
    csr = MB.build(g, None, "gcn")
    H, W = rng.standard_normal((7, 6)), rng.standard_normal((6, 2))
    a = Lr.gcn_forward(csr, H, W, False)["Z"]
    b = Lr.aggregate(csr, H @ W)
    assert rel(a, b) < 1e-12


def test_theory_model_gradient_closed_form():
    """Appendix C.1: one hidden layer, fixed output weights a, sub-GCN mask."""
    n, d, d1, m = 6, 3, 8, 2
    g = erdos_renyi(n, 8, seed=11)
    csr = MB.build(g, None, "theory")
    Abar = MB.dense(csr)
    rng = np.random.default_rng(6)
    X = rng.standard_normal((n, d))
    Theta = rng.standard_normal((d, d1))
    a = rng.choice([-1.0, 1.0], size=d1)
    y = rng.standard_normal(n)
    idx, offs = P.partition(d1, m, 21)
    Dj = idx[offs[0]:offs[1]]
    Xh = Abar @ X
    # generic two-layer chain: hidden GCN layer on the block's columns, then
    # a linear GCN layer with weights a_r / sqrt(d1) on the same block.
    W0 = Theta[:, Dj]
    W1 = (a[Dj] / np.sqrt(d1))[:, None]
    f0 = Lr.gcn_forward(csr, X, W0, True)
    f1 = Lr.gcn_forward(csr, f0["H_out"], W1, False)
    yhat = f1["H_out"][:, 0]
    b1 = Lr.gcn_backward(csr, f0["H_out"], f1, W1, (yhat - y)[:, None], False)
    b0 = Lr.gcn_backward(csr, X, f0, W0, b1["dH"], True, need_dH=False)
    # closed form, term by term: sum_i sum_i' (yhat_i - y_i) Abar_ii' M_r a_r xhat_i' 1{<theta_r, xhat_i'> >= 0}
    mask = np.zeros(d1)
    mask[Dj] = 1.0
    want = np.zeros((d, d1))
    for r in range(d1):
        for i in range(n):
            for ip in range(n):
                if Xh[ip] @ Theta[:, r] >= 0:
                    want[:, r] += ((yhat[i] - y[i]) * Abar[i, ip] * mask[r] * a[r]
                                   * Xh[ip]) / np.sqrt(d1)
    assert rel(b0["dW"], want[:, Dj]) < 1e-12
    others = [r for r in range(d1) if r not in Dj]
    assert np.all(want[:, others] == 0.0)


def test_sgd_and_slices():
    rng = np.random.default_rng(8)
    W, dW = rng.standard_normal((4, 5)), rng.standard_normal((4, 5))
    assert np.array_equal(Lr.sgd(W, dW, 0.0), W)
    T = rng.standard_normal((6, 7))
    r, c = [1, 4], [0, 2, 6]
    s = Lr.gather_slice(T, r, c)
    assert s.shape == (2, 3) and s[1, 2] == T[4, 6]
    assert np.array_equal(Lr.subagg(T, r, c, s), T)  # round trip
    z = Lr.subagg(T, r, c, np.zeros((2, 3)))
    mask = np.ones_like(T, dtype=bool)
    mask[np.ix_(r, c)] = False
    assert np.array_equal(z[mask], T[mask]) and np.all(z[np.ix_(r, c)] == 0)
    assert np.array_equal(Lr.gather_slice(T, None, c), T[:, c])


# ---- options of the layers: association order, rounded operands, masks ----

def test_round_bf16_matches_torch_conversion():
    """The bf16-input variant's operand rounding against torch's own
    float -> bfloat16 conversion (round to nearest even): random values over
    many binades, exact ties (to even, both directions), values that round
    up across a binade, the largest finite values, subnormals, zeros and
    infinities."""
    import torch
    rng = np.random.default_rng(11)
    x = np.concatenate([
        rng.standard_normal(20000) * np.exp(rng.uniform(-30, 30, 20000)),
        np.float32(1.0) + np.arange(-40, 40, dtype=np.float32) * np.float32(2.0 ** -9),
        [1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, 1.0 - 2.0 ** -9, 2.0 - 2.0 ** -9,
         3.3895313892515355e38, 3.4028234663852886e38, 1e-40, -1e-40, 0.0, -0.0,
         np.inf, -np.inf]]).astype(np.float32)
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = Lr.round_bf16(x)
    assert np.array_equal(got, want)
    # ties go to the even neighbour: 1 + 2^-8 lies halfway between 1 and
    # 1 + 2^-7 and rounds to 1; 1 + 3 2^-8 rounds up to 1 + 2^-6
    assert Lr.round_bf16(1.0 + 2.0 ** -8) == 1.0
    assert Lr.round_bf16(1.0 + 3 * 2.0 ** -8) == 1.0 + 2.0 ** -6
    assert np.isnan(Lr.round_bf16(np.nan))


def _rect_csr(seed, n, n_in):
    """A random rectangular aggregation matrix (rows n, columns n_in) with
    its explicit transpose, as a layer-sampled mini-batch stores it."""
    import scipy.sparse as sps
    rng = np.random.default_rng(seed)
    A = sps.random(n, n_in, density=0.3, random_state=seed, format="csr", dtype=np.float64)
    A.data = A.data.astype(np.float32).astype(np.float64)
    At = A.T.tocsr()
    At.sort_indices()
    A.sort_indices()
    return dict(n=n, n_in=n_in, nnz=A.nnz, rowptr=A.indptr, col=A.indices,
                val=A.data.astype(np.float32), t_rowptr=At.indptr, t_col=At.indices,
                t_val=At.data.astype(np.float32)), rng


@pytest.mark.parametrize("rect", [False, True])
def test_gcn_xform_order_equals_agg_order_in_fp64(tiny, rect):
    """(Abar H) W and Abar (H W), forward and backward, agree to rounding in
    fp64 (eq. (2) fixes no association order), square and rectangular."""
    if rect:
        csr, rng = _rect_csr(4, 5, 9)
    else:
        g, rng = tiny
        csr = MB.build(g, None, "gcn")
    n, n_in = csr["n"], csr.get("n_in", csr["n"])
    H, W = rng.standard_normal((n_in, 6)), rng.standard_normal((6, 3))
    dHo = rng.standard_normal((n, 3))
    fa = Lr.gcn_forward(csr, H, W, True, order="agg")
    fx = Lr.gcn_forward(csr, H, W, True, order="xform")
    assert rel(fx["Z"], fa["Z"]) < 1e-12
    ba = Lr.gcn_backward(csr, H, fa, W, dHo, True, order="agg")
    bx = Lr.gcn_backward(csr, H, fa, W, dHo, True, order="xform")
    assert rel(bx["dW"], ba["dW"]) < 1e-12 and rel(bx["dH"], ba["dH"]) < 1e-12
    with pytest.raises(ValueError):
        Lr.gcn_forward(csr, H, W, True, order="both")


def test_rounded_products_closed_form():
    """With no edges the GCN matrix is the identity, so a rounded layer is
    round(H) round(W) exactly: 1 + 2^-10 rounds to 1, 3 is exact, so
    Z = 3 where fp64 gives 3 (1 + 2^-10); SAGE's self term the same; the
    backward's products round their operands too (dZ = 1 + 2^-9 rounds to
    1 + 2^-8 ... to even: 1)."""
    g = graph_from_edges(1, [])
    csr = MB.build(g, None, "gcn")
    H, W = np.array([[1.0 + 2.0 ** -10]]), np.array([[3.0]])
    for order in ("agg", "xform"):
        f = Lr.gcn_forward(csr, H, W, False, rnd=Lr.round_bf16, order=order)
        assert f["Z"][0, 0] == 3.0
        assert Lr.gcn_forward(csr, H, W, False, order=order)["Z"][0, 0] == 3.0 * (1 + 2.0 ** -10)
        b = Lr.gcn_backward(csr, H, f, W, np.array([[1.0 + 2.0 ** -9]]), False,
                            rnd=Lr.round_bf16, order=order)
        assert b["dW"][0, 0] == 1.0 and b["dH"][0, 0] == 3.0
    cs = MB.build(g, None, "sage")
    f = Lr.sage_forward(cs, H, W, W, False, rnd=Lr.round_bf16)
    assert f["Z"][0, 0] == 3.0 and np.array_equal(f["AH"], [[0.0]])


@pytest.mark.parametrize("kind", ["gcn", "sage"])
def test_rounded_layer_within_bf16_error_bound(tiny, kind):
    """Each rounded operand carries a relative error of at most 2^-8 (plus
    2^-24 from its fp32 form), so every entry of a rounded product differs
    from the exact one by at most (2^-7 + 2^-15) sum_k |a_ik||b_kj|; and the
    rounding is not the identity (the result differs from fp64)."""
    g, rng = tiny
    csr = MB.build(g, None, kind)
    H, W1, W2 = (rng.standard_normal((7, 6)), rng.standard_normal((6, 4)),
                 rng.standard_normal((6, 4)))
    u = 2.0 ** -7 + 2.0 ** -15
    if kind == "gcn":
        f = Lr.gcn_forward(csr, H, W1, False, rnd=Lr.round_bf16)
        e = Lr.gcn_forward(csr, H, W1, False)
        bound = u * (np.abs(e["AH"]) @ np.abs(W1))
    else:
        f = Lr.sage_forward(csr, H, W1, W2, False, rnd=Lr.round_bf16)
        e = Lr.sage_forward(csr, H, W1, W2, False)
        bound = u * (np.abs(H) @ np.abs(W1) + np.abs(e["AH"]) @ np.abs(W2))
    assert np.all(np.abs(f["Z"] - e["Z"]) <= bound)
    assert np.any(f["Z"] != e["Z"])


@pytest.mark.parametrize("kind", ["gcn", "sage"])
def test_mask_replaces_the_relu_derivative(tiny, kind):
    """mask = 1[Z > 0] reproduces the backward bit for bit; flipping one
    decision (i, f) changes the weight gradient by exactly the outer product
    of that row's input with dH_out[i, f] in column f (the chain rule with
    that one derivative changed), and nothing else."""
    g, rng = tiny
    csr = MB.build(g, None, kind)
    H, W1, W2 = (rng.standard_normal((7, 5)), rng.standard_normal((5, 4)),
                 rng.standard_normal((5, 4)))
    dHo = rng.standard_normal((7, 4))
    if kind == "gcn":
        f = Lr.gcn_forward(csr, H, W1, True)
        run = lambda m: Lr.gcn_backward(csr, H, f, W1, dHo, True, mask=m)
        X = f["AH"]
        grad = lambda b: b["dW"]
    else:
        f = Lr.sage_forward(csr, H, W1, W2, True)
        run = lambda m: Lr.sage_backward(csr, H, f, W1, W2, dHo, True, mask=m)
        X = np.concatenate([H, f["AH"]], axis=1)
        grad = lambda b: np.concatenate([b["dW_self"], b["dW_neigh"]])
    base = run(None)
    same = run(f["Z"] > 0)
    for k in base:
        assert np.array_equal(base[k], same[k])
    mask = f["Z"] > 0
    i, c = 3, 2
    mask[i, c] = not mask[i, c]
    flip = run(mask)
    delta = grad(flip) - grad(base)
    sign = 1.0 if mask[i, c] else -1.0
    want = np.zeros_like(delta)
    want[:, c] = sign * X[i] * dHo[i, c]
    assert np.max(np.abs(delta - want)) <= 1e-12 * np.max(np.abs(grad(base)))
    with pytest.raises(ValueError):
        run(mask[:, :2])
