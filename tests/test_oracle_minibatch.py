"""Pins of the oracle's mini-batch construction and normalisation.

Checked against brute force on dense matrices and against spectral facts:
the self-looped symmetric normalisation has the eigenvector D~^{1/2} 1 with
eigenvalue 1 and spectrum in (-1, 1]; the theory form I + D^-1/2 A D^-1/2
has spectrum in [0, 2] (Appendix C.2), reaching 2 on a bipartite graph;
mean-aggregation rows sum to one.
"""

import numpy as np
import pytest

from gist_synth.graphs import Graph, _csr_from_undirected, erdos_renyi, sbm
from oracle import minibatch as MB


def graph_from_edges(n, edges, cluster_sizes=None):
    u = [a for a, b in edges]
    v = [b for a, b in edges]
    rowptr, col = _csr_from_undirected(n, u, v)
    if cluster_sizes is None:
        cptr = np.array([0, n], dtype=np.int64)
    else:
        cptr = np.concatenate([[0], np.cumsum(cluster_sizes)]).astype(np.int64)
    return Graph(n, rowptr, col, cptr, np.arange(n, dtype=np.int32))


def dense_adj(g):
    a = np.zeros((g.n, g.n))
    for i in range(g.n):
        for e in range(g.rowptr[i], g.rowptr[i + 1]):
            a[i, g.col[e]] = 1.0
    return a


@pytest.fixture(scope="module")
def small():
    # 3 clusters of sizes 5, 4, 3 on an ER graph with an isolated node.
    g = erdos_renyi(12, 18, seed=5, clusters=3)
    return g


def induced_dense(g, nodes):
    return dense_adj(g)[np.ix_(nodes, nodes)]


@pytest.mark.parametrize("sel", [None, [0], [2, 0], [1, 1, 2]])
def test_gcn_matches_dense_brute_force(small, sel):
    csr = MB.build(small, sel, "gcn")
    nodes = csr["node_map"]
    assert list(nodes) == sorted(nodes)
    A = induced_dense(small, nodes)
    At = A + np.eye(len(nodes))
    dinv = np.diag(1.0 / np.sqrt(At.sum(axis=1)))
    want = dinv @ At @ dinv
    got = MB.dense(csr)
    assert ((got != 0) == (want != 0)).all()
    nz = want != 0
    assert np.max(np.abs(got[nz] - want[nz]) / want[nz]) <= 2.0 ** -24
    # bitwise symmetric
    assert (got == got.T).all()
    # columns ascending and strictly increasing per row
    for i in range(csr["n"]):
        c = csr["col"][csr["rowptr"][i]:csr["rowptr"][i + 1]]
        assert (np.diff(c) > 0).all()


def test_gcn_eigenvector_and_spectrum(small):
    csr = MB.build(small, None, "gcn")
    A = MB.dense(csr)
    dt = (A != 0).sum(axis=1).astype(float)  # 1 + degree (self-loop included)
    v = np.sqrt(dt)
    assert np.allclose(A @ v, v, rtol=1e-6, atol=0)
    ev = np.linalg.eigvalsh(A)
    assert ev.max() == pytest.approx(1.0, abs=1e-6)
    assert ev.min() > -1.0 - 1e-6


def test_theory_form_spectrum():
    g = erdos_renyi(14, 30, seed=9)
    ev = np.linalg.eigvalsh(MB.dense(MB.build(g, None, "theory")))
    assert ev.min() >= -1e-6 and ev.max() <= 2.0 + 1e-6
    # bipartite path graph reaches the upper end of the spectrum
    path = graph_from_edges(6, [(i, i + 1) for i in range(5)])
    ev = np.linalg.eigvalsh(MB.dense(MB.build(path, None, "theory")))
    assert ev.max() == pytest.approx(2.0, abs=1e-6)
    # diagonal is exactly one
    A = MB.dense(MB.build(path, None, "theory"))
    assert (np.diag(A) == 1.0).all()


def test_sage_rows_and_transpose(small):
    csr = MB.build(small, [0, 1], "sage")
    A = MB.dense(csr)
    nodes = csr["node_map"]
    Ai = induced_dense(small, nodes)
    deg = Ai.sum(axis=1)
    assert ((A != 0) == (Ai != 0)).all()
    assert np.allclose(A.sum(axis=1)[deg > 0], 1.0, atol=1e-6)
    assert (A.sum(axis=1)[deg == 0] == 0).all()
    assert (np.diag(A) == 0).all()
    assert (MB.dense(csr, transpose=True) == A.T).all()


def test_isolated_node_rows():
    g = graph_from_edges(4, [(0, 1), (1, 2)])  # node 3 isolated
    gcn = MB.build(g, None, "gcn")
    assert gcn["rowptr"][4] - gcn["rowptr"][3] == 1  # only the self-loop
    assert gcn["val"][-1] == np.float32(1.0)
    sage = MB.build(g, None, "sage")
    assert sage["rowptr"][4] == sage["rowptr"][3]  # empty row


def test_all_clusters_equals_full_graph(small):
    for norm in MB.NORMS:
        a = MB.build(small, None, norm)
        b = MB.build(small, [2, 1, 0], norm)
        for k in ("rowptr", "col", "val", "node_map"):
            assert np.array_equal(a[k], b[k])


def test_induced_edges_exact_on_sbm():
    g = sbm(600, 6, 20.0, 0.9, seed=3)
    csr = MB.build(g, [4, 1], "gcn")
    nodes = csr["node_map"]
    want = np.concatenate([np.arange(g.cluster_ptr[1], g.cluster_ptr[2]),
                           np.arange(g.cluster_ptr[4], g.cluster_ptr[5])])
    assert np.array_equal(nodes, want)
    A = induced_dense(g, nodes) + np.eye(len(nodes))
    assert ((MB.dense(csr) != 0) == (A != 0)).all()


def test_selection_errors(small):
    with pytest.raises(ValueError):
        MB.build(small, [], "gcn")
    with pytest.raises(ValueError):
        MB.build(small, [3], "gcn")
    with pytest.raises(ValueError):
        MB.build(small, [-1], "gcn")
