"""Seeded random graphs in the layout the library's host API takes.

A :class:`Graph` is a simple undirected graph without self-loops stored as a
symmetric CSR adjacency (``rowptr`` int64[n+1], ``col`` int32[nnz], columns
strictly ascending within each row) plus a clustering (``cluster_ptr``
int64[c+1], ``cluster_nodes`` int32[n]).  Node ids are block-contiguous, so
cluster ``b`` is the id range ``[cluster_ptr[b], cluster_ptr[b+1])`` -- the
order a METIS-reordered graph would have (the paper clusters with METIS,
Section 2, and ClusterGCN-style mini-batches are unions of clusters).

Three families cover the workloads' degree structure:

* ``erdos_renyi``: G(n, M), exactly M distinct edges (concentrated degrees).
* ``chung_lu``: expected-degree power law (heavy-tailed rows, hub nodes).
* ``sbm``: stochastic block model with equal blocks, a fixed intra-block
  probability and a fixed number of uniformly placed inter-block edges.
"""

from dataclasses import dataclass

import numpy as np
import scipy.sparse as sp

from .seeds import STREAM_GRAPH, generator


@dataclass
class Graph:
    n: int
    rowptr: np.ndarray          # int64[n+1]
    col: np.ndarray             # int32[nnz], ascending per row
    cluster_ptr: np.ndarray     # int64[c+1]
    cluster_nodes: np.ndarray   # int32[n]

    @property
    def nnz(self):
        return int(self.rowptr[-1])

    @property
    def n_clusters(self):
        return int(self.cluster_ptr.shape[0] - 1)

    def degrees(self):
        return np.diff(self.rowptr)


def _csr_from_undirected(n, u, v):
    """Symmetric CSR (int64 rowptr, int32 col, ascending) from edges u<v."""
    u = np.asarray(u, dtype=np.int64)
    v = np.asarray(v, dtype=np.int64)
    rows = np.concatenate([u, v])
    cols = np.concatenate([v, u])
    data = np.ones(rows.shape[0], dtype=np.int8)
    a = sp.csr_matrix((data, (rows, cols)), shape=(n, n))
    a.sum_duplicates()
    a.sort_indices()
    rowptr = a.indptr.astype(np.int64)
    col = a.indices.astype(np.int32)
    return rowptr, col


def _single_cluster(n):
    return (np.array([0, n], dtype=np.int64), np.arange(n, dtype=np.int32))


def _dedupe_in_order(keys):
    """Unique keys, keeping first occurrences in draw order."""
    _, first = np.unique(keys, return_index=True)
    return keys[np.sort(first)]


def erdos_renyi(n, n_edges, seed, clusters=None):
    """G(n, M): ``n_edges`` distinct undirected edges drawn uniformly.

    ``clusters``: optional number of equal contiguous id blocks to expose as
    the clustering (default: one cluster = the whole graph).
    """
    rng = generator(seed, STREAM_GRAPH, 1)
    keys = np.zeros(0, dtype=np.int64)
    while keys.shape[0] < n_edges:
        need = n_edges - keys.shape[0]
        a = rng.integers(0, n, size=2 * need + 16, dtype=np.int64)
        b = rng.integers(0, n, size=2 * need + 16, dtype=np.int64)
        keep = a != b
        lo = np.minimum(a[keep], b[keep])
        hi = np.maximum(a[keep], b[keep])
        keys = _dedupe_in_order(np.concatenate([keys, lo * n + hi]))
    keys = keys[:n_edges]
    rowptr, col = _csr_from_undirected(n, keys // n, keys % n)
    if clusters is None:
        cptr, cnodes = _single_cluster(n)
    else:
        cptr, cnodes = _equal_blocks(n, clusters)
    return Graph(n, rowptr, col, cptr, cnodes)


def chung_lu(n, gamma, mean_degree, seed):
    """Chung-Lu graph with expected degrees w_i proportional to (i+1)^(-1/(gamma-1)).

    The weights are scaled to mean ``mean_degree``; each pair i<j is an edge
    independently with probability min(1, w_i w_j / sum(w)).  Node 0 is the
    largest hub.  One cluster (the full graph).
    """
    rng = generator(seed, STREAM_GRAPH, 2)
    w = (np.arange(n, dtype=np.float64) + 1.0) ** (-1.0 / (gamma - 1.0))
    w *= mean_degree * n / w.sum()
    s = w.sum()
    us, vs = [], []
    chunk = max(1, (1 << 22) // n)
    jj = np.arange(n, dtype=np.int64)
    for a in range(0, n, chunk):
        b = min(n, a + chunk)
        ii = np.arange(a, b, dtype=np.int64)
        p = np.minimum(1.0, np.outer(w[a:b], w) / s)
        r = rng.random((b - a, n))
        hit = (r < p) & (jj[None, :] > ii[:, None])
        ri, cj = np.nonzero(hit)
        us.append(ii[ri])
        vs.append(cj.astype(np.int64))
    u = np.concatenate(us)
    v = np.concatenate(vs)
    rowptr, col = _csr_from_undirected(n, u, v)
    cptr, cnodes = _single_cluster(n)
    return Graph(n, rowptr, col, cptr, cnodes)


def _equal_blocks(n, blocks):
    base, rem = divmod(n, blocks)
    sizes = np.full(blocks, base, dtype=np.int64)
    sizes[:rem] += 1
    ptr = np.zeros(blocks + 1, dtype=np.int64)
    np.cumsum(sizes, out=ptr[1:])
    return ptr, np.arange(n, dtype=np.int32)


def sbm(n, blocks, mean_degree, intra_frac, seed):
    """Stochastic block model with ``blocks`` equal contiguous blocks.

    Intra-block pairs are edges independently with probability
    p_in = intra_frac * mean_degree / (n/blocks - 1); then
    round((1-intra_frac) * mean_degree * n / 2) distinct inter-block edges are
    drawn uniformly over cross-block pairs.  The blocks are the clusters.
    """
    rng = generator(seed, STREAM_GRAPH, 3)
    ptr, cnodes = _equal_blocks(n, blocks)
    sizes = np.diff(ptr)
    p_in = intra_frac * mean_degree / (n / blocks - 1.0)
    us, vs = [], []
    for s in np.unique(sizes):
        bids = np.nonzero(sizes == s)[0]
        iu, ju = np.triu_indices(int(s), 1)
        npairs = iu.shape[0]
        step = max(1, (1 << 24) // max(1, npairs))
        for a in range(0, bids.shape[0], step):
            bb = bids[a:a + step]
            hit = rng.random((bb.shape[0], npairs), dtype=np.float32) < p_in
            bi, pi = np.nonzero(hit)
            start = ptr[bb][bi]
            us.append(start + iu[pi])
            vs.append(start + ju[pi])
    n_inter = int(round((1.0 - intra_frac) * mean_degree * n / 2.0))
    keys = np.zeros(0, dtype=np.int64)
    while keys.shape[0] < n_inter:
        need = n_inter - keys.shape[0]
        a = rng.integers(0, n, size=need + need // 8 + 16, dtype=np.int64)
        b = rng.integers(0, n, size=need + need // 8 + 16, dtype=np.int64)
        ba = np.searchsorted(ptr, a, side="right") - 1
        bb_ = np.searchsorted(ptr, b, side="right") - 1
        keep = ba != bb_
        lo = np.minimum(a[keep], b[keep])
        hi = np.maximum(a[keep], b[keep])
        keys = _dedupe_in_order(np.concatenate([keys, lo * n + hi]))
    keys = keys[:n_inter]
    us.append(keys // n)
    vs.append(keys % n)
    u = np.concatenate(us)
    v = np.concatenate(vs)
    rowptr, col = _csr_from_undirected(n, u, v)
    return Graph(n, rowptr, col, ptr, cnodes)
