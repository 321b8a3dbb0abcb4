"""Sub-GCN layer forward/backward, loss, SGD, slice gather and ``subAgg`` in fp64.

Paper:

* eq. (1) and eq. (2): H_{l+1} = sigma(Abar H_l Theta_l) for the full and the
  sub-GCN layer (no rescaling of the sub-GCN); the last layer's activation
  is the identity and the loss is unchanged by GIST (Section 2.1);
* GraphSAGE (Section 3, related work): the aggregated neighbourhood is
  concatenated with the node's own representation.  With the mean
  aggregator this is Z = H Theta_self + (D^-1 A) H Theta_neigh, i.e. the
  concatenation [H | Abar H] times [Theta_self; Theta_neigh];
* ``subTrain`` is one SGD step (Section 2.2); the theory writes the same
  update as theta <- theta - eta dL/dtheta (eq. "GIST_procedure");
* Theta^(i)_l = rows D^(i)_l and columns D^(i)_{l+1} of Theta_l (Section 2.1);
* ``subAgg`` replaces those entries of the global Theta with the trained
  slice and leaves every other entry unchanged (Section 2.2).

The backward pass is the chain rule of the forward written out: the ReLU
derivative is 1[Z > 0]; the aggregation's adjoint is the transpose of the
stored matrix (no symmetry is assumed).  Matrix products use NumPy / SciPy
primitives in fp64; nothing is blocked, fused or reordered beyond the
definitions.
"""

import numpy as np
import scipy.sparse as sp


def as_f64(x):
    return np.asarray(x, dtype=np.float64)


def adjacency(csr, transpose=False):
    """The stored aggregation matrix (or its explicit transpose) as fp64 CSR.

    A matrix with ``n_in`` (columns) different from ``n`` (rows) aggregates
    from one node set into another (a layer-sampled mini-batch); its stored
    transpose has the swapped shape."""
    key = "t_" if transpose else ""
    n = csr["n"]
    n_in = csr.get("n_in", n)
    shape = (n_in, n) if transpose else (n, n_in)
    return sp.csr_matrix((csr[key + "val"].astype(np.float64),
                          csr[key + "col"].astype(np.int64),
                          csr[key + "rowptr"].astype(np.int64)), shape=shape)


def aggregate(csr, H):
    """Abar H (eq. (1)): row i is sum_j Abar_ij H_j."""
    return adjacency(csr) @ as_f64(H)


def aggregate_transposed(csr, G):
    """Abar^T G, the adjoint of :func:`aggregate` (transpose of the stored matrix)."""
    return adjacency(csr).T @ as_f64(G)


def relu(z):
    return np.maximum(z, 0.0)


def gcn_forward(csr, H, W, act):
    """GCN layer, eq. (2): Z = (Abar H) W, H' = ReLU(Z) if ``act`` else Z."""
    AH = aggregate(csr, H)
    Z = AH @ as_f64(W)
    return dict(AH=AH, Z=Z, H_out=relu(Z) if act else Z)


def sage_forward(csr, H, W_self, W_neigh, act):
    """GraphSAGE-mean layer: Z = H W_self + (D^-1 A H) W_neigh."""
    H = as_f64(H)
    AH = aggregate(csr, H)
    Z = H @ as_f64(W_self) + AH @ as_f64(W_neigh)
    return dict(AH=AH, Z=Z, H_out=relu(Z) if act else Z)


def _dz(Z, dH_out, act):
    dH_out = as_f64(dH_out)
    return dH_out * (Z > 0.0) if act else dH_out


def gcn_backward(csr, H, fwd, W, dH_out, act, need_dH=True):
    """Gradients of the GCN layer: dW = (Abar H)^T dZ, dH = Abar^T (dZ W^T).

    Abar^T is the transpose of the stored matrix, formed here.
    """
    dZ = _dz(fwd["Z"], dH_out, act)
    out = dict(dZ=dZ, dW=fwd["AH"].T @ dZ)
    if need_dH:
        dP = dZ @ as_f64(W).T
        out["dH"] = aggregate_transposed(csr, dP)
    return out


def sage_backward(csr, H, fwd, W_self, W_neigh, dH_out, act, need_dH=True):
    """Gradients of the SAGE-mean layer.

    dW_self = H^T dZ, dW_neigh = (Abar H)^T dZ,
    dH = dZ W_self^T + Abar^T (dZ W_neigh^T), with Abar^T the stored transpose.
    """
    H = as_f64(H)
    dZ = _dz(fwd["Z"], dH_out, act)
    out = dict(dZ=dZ, dW_self=H.T @ dZ, dW_neigh=fwd["AH"].T @ dZ)
    if need_dH:
        dP = dZ @ as_f64(W_neigh).T
        if "t_val" in csr:
            agg_t = adjacency(csr, transpose=True) @ dP
        else:
            agg_t = aggregate_transposed(csr, dP)
        out["dH"] = dZ @ as_f64(W_self).T + agg_t
    return out


def softmax_xent(Z, labels):
    """Mean softmax cross-entropy and its gradient (softmax - onehot) / n."""
    Z = as_f64(Z)
    n = Z.shape[0]
    labels = np.asarray(labels, dtype=np.int64)
    if n == 0:
        return 0.0, np.zeros_like(Z)
    if labels.min() < 0 or labels.max() >= Z.shape[1]:
        raise ValueError("label out of range")
    zmax = Z.max(axis=1, keepdims=True)
    lse = zmax[:, 0] + np.log(np.exp(Z - zmax).sum(axis=1))
    loss = float(np.mean(lse - Z[np.arange(n), labels]))
    P = np.exp(Z - lse[:, None])
    P[np.arange(n), labels] -= 1.0
    return loss, P / n


def sgd(W, dW, lr):
    """One SGD step, W - lr dW."""
    return as_f64(W) - float(lr) * as_f64(dW)


def gather_slice(theta, rows, cols):
    """Theta[rows, cols] (None: all rows / all columns), Section 2.1."""
    theta = np.asarray(theta)
    r = np.arange(theta.shape[0]) if rows is None else np.asarray(rows)
    c = np.arange(theta.shape[1]) if cols is None else np.asarray(cols)
    return theta[np.ix_(r, c)].copy()


def subagg(theta, rows, cols, slice_):
    """Copy of ``theta`` with entries (rows x cols) replaced by ``slice_``."""
    out = np.array(theta, copy=True)
    r = np.arange(out.shape[0]) if rows is None else np.asarray(rows)
    c = np.arange(out.shape[1]) if cols is None else np.asarray(cols)
    out[np.ix_(r, c)] = slice_
    return out
