"""LADIES layer-wise sampled mini-batches, the node sampling GIST is paired
with instead of graph partitioning (Section 5.4 and Appendix A.6: a vanilla GCN of 2 or 3 layers, LADIES in place of
``Cluster``).

TEST INFRASTRUCTURE ONLY (see :mod:`oracle`): plain fp64 loops, no shared
code with the library.

LADIES (Zou et al., "Layer-Dependent Importance Sampling for Training Deep
and Large Graph Convolutional Networks", NeurIPS 2019) builds one sampled
aggregation matrix per layer, from the output layer down.  With P the
normalised adjacency and Q^(l) the rows of the nodes kept at layer l:

* the layer-dependent importance of node j is the squared norm of column j
  of Q^(l) P, normalised to a distribution p^(l-1) over the graph;
* s nodes are drawn from it independently (with replacement);
* the sampled matrix is Q^(l) P S^(l-1), S^(l-1) diagonal with 1/(s p_j) on
  the kept nodes, and its rows are normalised to sum to one.

The GIST paper gives no detail beyond using LADIES, so the following
readings fix what the sampler computes, such that two independent
implementations agree bit for bit:

* P is the full-graph GCN matrix of eq. (1) (``oracle.minibatch.build`` with
  ``clusters=None``, "gcn"); its fp32 values are widened to fp64.
* Node sets V_0 ⊇ V_1 ⊇ ... ⊇ V_L, where V_L (the output nodes) is given,
  ascending and distinct.  Layer l (0-based) aggregates from V_l into
  V_{l+1}; sampling runs l = L-1, ..., 0.
* q_j = sum over i in V_{l+1}, i ascending, of P_ij^2 (fp64, accumulated in
  that order); Q = sum of q_j over j ascending; p_j = q_j / Q.
* One SplitMix64 stream (``oracle.partition.SplitMix64``) seeded ``seed``
  serves every layer, layer L-1 first, s outputs per layer.  Output x gives
  u = (x >> 11) * 2^-53 and t = u * Q; the drawn node is the smallest j
  whose prefix sum C_j = q_0 + ... + q_j (ascending j) exceeds t; if t
  rounded up to Q or beyond, the largest j with q_j > 0.
* V_l = the distinct drawn nodes together with V_{l+1} (as LADIES keeps the
  output nodes so that every row keeps its self-loop), ascending.
* The sampled matrix has rows V_{l+1} and columns V_l; row i holds every
  stored entry (i, j) of P with j in V_l, in ascending j, value
  w_ij = P_ij / (s p_j) (s p_j formed as float(s) * p_j, with s taken as 1
  when s = 0: no draws, V_l = V_{l+1}); each row is divided by its sum
  taken in ascending j, and the quotient is rounded once to fp32.  A node
  of V_l is weighted once however often it was drawn.
* The transpose (rows V_l, columns V_{l+1}) is stored for the backward pass.
* No output node (V_L empty): every V_l is empty and nothing is drawn.
"""

import numpy as np

from .partition import SplitMix64


def _check_batch(n, batch):
    b = np.asarray(batch, dtype=np.int64)
    if b.ndim != 1:
        raise ValueError("batch must be a vector of node ids")
    if b.size and (b.min() < 0 or b.max() >= n):
        raise ValueError("batch node id out of range")
    if b.size > 1 and np.any(np.diff(b) <= 0):
        raise ValueError("batch must be ascending and distinct")
    return b


def importance(P, rows):
    """q_j = sum_{i in rows} P_ij^2, accumulated row by row in the given order."""
    q = np.zeros(P["n"], dtype=np.float64)
    rp, col, val = P["rowptr"], P["col"], P["val"]
    for i in rows:
        for e in range(int(rp[i]), int(rp[i + 1])):
            a = float(val[e])
            q[int(col[e])] += a * a
    return q


def draw(q, s, rng):
    """s i.i.d. draws from p = q / sum(q) by inverse CDF on the prefix sums."""
    C = np.cumsum(q)          # sequential prefix sums, ascending j
    Q = float(C[-1]) if C.size else 0.0
    if s == 0:
        return []
    if not Q > 0.0:
        raise ValueError("no node has positive importance")
    last = int(np.nonzero(q > 0.0)[0][-1])
    out = []
    for _ in range(s):
        u = float(rng.next() >> 11) * 2.0 ** -53
        t = u * Q
        j = int(np.searchsorted(C, t, side="right"))
        out.append(j if j < q.size else last)
    return out


def sampled_matrix(P, rows, cols, p, s):
    """Row-normalised Q P S restricted to rows x cols (both ascending).

    Returns (rowptr, col, val) with local column indices into ``cols``."""
    pos = {int(j): k for k, j in enumerate(cols)}
    rp, col, val = P["rowptr"], P["col"], P["val"]
    rowptr = [0]
    out_c, out_v = [], []
    for i in rows:
        ks, ws = [], []
        for e in range(int(rp[i]), int(rp[i + 1])):
            j = int(col[e])
            if j in pos:
                ks.append(pos[j])
                ws.append(float(val[e]) / (float(s) * float(p[j])))
        total = 0.0
        for w in ws:
            total += w
        out_c.extend(ks)
        out_v.extend(np.float32(w / total) for w in ws)
        rowptr.append(len(out_c))
    return (np.asarray(rowptr, dtype=np.int64), np.asarray(out_c, dtype=np.int32),
            np.asarray(out_v, dtype=np.float32))


def _transpose(n_rows, n_cols, rowptr, col, val):
    """Explicit transpose; entries of each transposed row in ascending column."""
    t_rows = [[] for _ in range(n_cols)]
    for i in range(n_rows):
        for e in range(int(rowptr[i]), int(rowptr[i + 1])):
            t_rows[int(col[e])].append((i, val[e]))
    t_rowptr = np.zeros(n_cols + 1, dtype=np.int64)
    t_col, t_val = [], []
    for j in range(n_cols):
        for i, v in t_rows[j]:
            t_col.append(i)
            t_val.append(v)
        t_rowptr[j + 1] = len(t_col)
    return t_rowptr, np.asarray(t_col, dtype=np.int32), np.asarray(t_val, dtype=np.float32)


def sample(P, batch, L, s, seed):
    """LADIES mini-batch for an L-layer GCN.

    ``P``: the full-graph GCN CSR dict; ``batch``: output nodes V_L.
    Returns dict(nodes=[V_0, ..., V_L] (int64 arrays), layers=[layer dicts
    for l = 0..L-1]); layer l is a rectangular CSR with ``n`` = |V_{l+1}|
    rows, ``n_in`` = |V_l| columns, ``rowptr``/``col``/``val`` and the
    transpose ``t_rowptr``/``t_col``/``t_val``, plus ``p`` (the layer's
    distribution over all nodes) and ``draws`` (the drawn node ids).
    """
    n = int(P["n"])
    if L < 1 or s < 0:
        raise ValueError("L >= 1 and s >= 0 required")
    V = [None] * (L + 1)
    V[L] = _check_batch(n, batch)
    layers = [None] * L
    rng = SplitMix64(seed)
    for l in range(L - 1, -1, -1):
        out_nodes = V[l + 1]
        if out_nodes.size == 0:
            V[l] = out_nodes
            layers[l] = dict(n=0, n_in=0, nnz=0, rowptr=np.zeros(1, np.int64),
                             col=np.zeros(0, np.int32), val=np.zeros(0, np.float32),
                             t_rowptr=np.zeros(1, np.int64), t_col=np.zeros(0, np.int32),
                             t_val=np.zeros(0, np.float32), p=np.zeros(n), draws=[])
            continue
        q = importance(P, out_nodes)
        Q = float(np.cumsum(q)[-1])
        p = q / Q
        drawn = draw(q, s, rng)
        V[l] = np.array(sorted(set(drawn) | set(int(i) for i in out_nodes)), dtype=np.int64)
        rowptr, col, val = sampled_matrix(P, out_nodes, V[l], p, max(s, 1))
        t_rowptr, t_col, t_val = _transpose(out_nodes.size, V[l].size, rowptr, col, val)
        layers[l] = dict(n=int(out_nodes.size), n_in=int(V[l].size), nnz=int(rowptr[-1]),
                         rowptr=rowptr, col=col, val=val, t_rowptr=t_rowptr, t_col=t_col,
                         t_val=t_val, p=p, draws=drawn)
    return dict(nodes=V, layers=layers)


def dense(layer, transpose=False):
    """A sampled layer matrix (or its stored transpose) as a dense fp64 array."""
    key = "t_" if transpose else ""
    shape = (layer["n_in"], layer["n"]) if transpose else (layer["n"], layer["n_in"])
    a = np.zeros(shape, dtype=np.float64)
    rp, col, val = layer[key + "rowptr"], layer[key + "col"], layer[key + "val"]
    for i in range(shape[0]):
        for e in range(int(rp[i]), int(rp[i + 1])):
            a[i, int(col[e])] += float(val[e])
    return a
