"""``Cluster`` mini-batch: induced subgraph of a union of clusters, normalised.

Paper: Section 2.2 (a mini-batch is one cluster or the union of several
clusters of the training graph), Algorithm 1 (``Cluster``), eq. (1) (the
aggregation matrix is the degree-normalised adjacency with self-loops) and
Appendix C.2 (the theory form I + D^-1/2 A D^-1/2).

Readings fixed here where the paper is silent:

* the mini-batch keeps every edge whose two ends are both selected, and
  degrees are those of this induced subgraph;
* local node order is ascending global id, columns ascend in every row;
* ``gcn``: value (i, j) = 1 / sqrt(Dt_i * Dt_j) with Dt = 1 + induced degree
  (self-loop included), computed in fp64 (exact integer product, correctly
  rounded sqrt and division) and rounded once to fp32;
* ``sage``: GraphSAGE with the mean aggregator, value (i, j) = 1 / deg_i,
  no self-loop, a node with no neighbour keeps an empty row; the transpose
  is returned explicitly for the backward pass;
* ``theory``: 1.0 on the diagonal, 1 / sqrt(deg_i * deg_j) off it.
"""

import numpy as np

NORMS = ("gcn", "sage", "theory")


def select_nodes(graph, clusters):
    """Ascending global ids of the union of ``clusters`` (None: all nodes)."""
    if clusters is None:
        return np.arange(graph.n, dtype=np.int64)
    clusters = np.asarray(clusters, dtype=np.int64)
    if clusters.size == 0:
        raise ValueError("empty cluster selection")
    if clusters.min() < 0 or clusters.max() >= graph.n_clusters:
        raise ValueError("cluster id out of range")
    parts = [graph.cluster_nodes[graph.cluster_ptr[c]:graph.cluster_ptr[c + 1]]
             for c in np.unique(clusters)]
    return np.unique(np.concatenate(parts).astype(np.int64))


def induced_edges(graph, nodes):
    """Local (row, col) pairs of every edge with both ends in ``nodes``."""
    n_b = nodes.shape[0]
    local = np.full(graph.n, -1, dtype=np.int64)
    local[nodes] = np.arange(n_b, dtype=np.int64)
    starts = graph.rowptr[nodes]
    lens = graph.rowptr[nodes + 1] - starts
    # positions of every stored neighbour of every selected node
    pos = np.repeat(starts - np.cumsum(lens) + lens, lens) + np.arange(lens.sum())
    rows = np.repeat(np.arange(n_b, dtype=np.int64), lens)
    cols = local[graph.col[pos]]
    keep = cols >= 0
    return rows[keep], cols[keep]


def _to_csr(n_b, rows, cols, vals):
    order = np.lexsort((cols, rows))
    rows, cols, vals = rows[order], cols[order], vals[order]
    rowptr = np.zeros(n_b + 1, dtype=np.int64)
    np.add.at(rowptr, rows + 1, 1)
    rowptr = np.cumsum(rowptr)
    return rowptr, cols.astype(np.int32), vals


def build(graph, clusters, norm):
    """Mini-batch CSR for the union of ``clusters`` (None: full graph).

    Returns a dict with ``n``, ``nnz``, ``rowptr`` (int64), ``col`` (int32),
    ``val`` (float32), ``node_map`` (local -> global, int64) and, for
    ``sage``, the transpose ``t_rowptr``, ``t_col``, ``t_val``.
    """
    if norm not in NORMS:
        raise ValueError(norm)
    nodes = select_nodes(graph, clusters)
    n_b = nodes.shape[0]
    r, c = induced_edges(graph, nodes)
    deg = np.bincount(r, minlength=n_b).astype(np.float64)
    out = dict(n=n_b, node_map=nodes)
    if norm == "gcn":
        dt = deg + 1.0
        diag = np.arange(n_b, dtype=np.int64)
        rows = np.concatenate([r, diag])
        cols = np.concatenate([c, diag])
        vals = (1.0 / np.sqrt(dt[rows] * dt[cols])).astype(np.float32)
    elif norm == "theory":
        diag = np.arange(n_b, dtype=np.int64)
        rows = np.concatenate([r, diag])
        cols = np.concatenate([c, diag])
        off = (1.0 / np.sqrt(deg[r] * deg[c])).astype(np.float32)
        vals = np.concatenate([off, np.ones(n_b, dtype=np.float32)])
    else:
        rows, cols = r, c
        vals = (1.0 / deg[r]).astype(np.float32)
    rowptr, col, val = _to_csr(n_b, rows, cols, vals)
    out.update(rowptr=rowptr, col=col, val=val, nnz=int(rowptr[-1]))
    if norm == "sage":
        trp, tcol, tval = _to_csr(n_b, cols, rows, vals)
        out.update(t_rowptr=trp, t_col=tcol, t_val=tval)
    return out


def dense(csr, transpose=False):
    """Expand a CSR dict to a dense fp64 matrix (for tiny graphs)."""
    n = csr["n"]
    key = "t_" if transpose else ""
    rp, col, val = csr[key + "rowptr"], csr[key + "col"], csr[key + "val"]
    a = np.zeros((n, n), dtype=np.float64)
    for i in range(n):
        for e in range(rp[i], rp[i + 1]):
            a[i, col[e]] += float(val[e])
    return a
