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


def round_bf16(x):
    """Operand rounding of the bf16-input variant: each value is taken to
    fp32 (round to nearest even, as the GPU holds it) and then to the
    nearest bfloat16 (8 significant bits, ties to even), returned in fp64.

    bfloat16 is the upper half of an IEEE fp32 word, so rounding to nearest
    even keeps the upper 16 bits after adding 0x7FFF plus the lowest kept bit
    (a carry into the exponent is the correct rounding up, up to infinity).
    NaN stays NaN."""
    f = np.asarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    out = r.astype(np.uint32).view(np.float32).astype(np.float64)
    return np.where(np.isnan(f), np.nan, out)


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


# Options shared by the layers below.
#
# ``rnd``: the rounding applied to every operand of a dense product, None for
# none (plain fp64).  ``round_bf16`` gives the bf16-input variant: the
# products' inputs are rounded to bfloat16 and the products are then formed
# exactly (in fp64 here; fp32 accumulation on the GPU).  The aggregation is
# not a dense product and is never rounded.
#
# ``order`` (GCN only): "agg" forms (Abar H) W, "xform" forms Abar (H W).  The
# two are equal in exact arithmetic (the association order is free, eq. (2)),
# but not once the operands are rounded, so a rounded oracle follows the
# order the GPU took.  The backward pass follows the same order: "agg"
# computes dW = (Abar H)^T dZ and dH = Abar^T (dZ W^T); "xform" computes
# T = Abar^T dZ, dW = H^T T and dH = T W^T.
#
# ``mask`` (backward): the ReLU derivative to use instead of 1[Z > 0] -- the
# decisions another evaluation of the same forward took.  A pre-activation
# within rounding distance of zero may fall on either side; with the other
# side's decisions the backward pass is the chain rule of that other,
# equally correct, forward.


def _rnd(rnd):
    return as_f64 if rnd is None else rnd


def gcn_forward(csr, H, W, act, rnd=None, order="agg"):
    """GCN layer, eq. (2): Z = (Abar H) W, H' = ReLU(Z) if ``act`` else Z."""
    r = _rnd(rnd)
    AH = aggregate(csr, H)
    if order == "xform":
        Z = aggregate(csr, r(H) @ r(W))
    elif order == "agg":
        Z = r(AH) @ r(W)
    else:
        raise ValueError("order is 'agg' or 'xform'")
    return dict(AH=AH, Z=Z, H_out=relu(Z) if act else Z)


def sage_forward(csr, H, W_self, W_neigh, act, rnd=None):
    """GraphSAGE-mean layer: Z = H W_self + (D^-1 A H) W_neigh."""
    r = _rnd(rnd)
    H = as_f64(H)
    AH = aggregate(csr, H)
    Z = r(H) @ r(W_self) + r(AH) @ r(W_neigh)
    return dict(AH=AH, Z=Z, H_out=relu(Z) if act else Z)


def _dz(Z, dH_out, act, mask=None):
    dH_out = as_f64(dH_out)
    if not act:
        return dH_out
    if mask is not None:
        mask = np.asarray(mask, dtype=bool)
        if mask.shape != np.shape(Z):
            raise ValueError("mask shape differs from the pre-activation's")
        return dH_out * mask
    return dH_out * (Z > 0.0)


def gcn_backward(csr, H, fwd, W, dH_out, act, need_dH=True, mask=None, rnd=None, order="agg"):
    """Gradients of the GCN layer: dW = (Abar H)^T dZ, dH = Abar^T (dZ W^T).

    Abar^T is the transpose of the stored matrix, formed here.
    """
    r = _rnd(rnd)
    dZ = _dz(fwd["Z"], dH_out, act, mask)
    if order == "xform":
        T = aggregate_transposed(csr, dZ)
        out = dict(dZ=dZ, dW=r(H).T @ r(T))
        if need_dH:
            out["dH"] = r(T) @ r(W).T
        return out
    if order != "agg":
        raise ValueError("order is 'agg' or 'xform'")
    out = dict(dZ=dZ, dW=r(fwd["AH"]).T @ r(dZ))
    if need_dH:
        dP = r(dZ) @ r(W).T
        out["dH"] = aggregate_transposed(csr, dP)
    return out


def sage_backward(csr, H, fwd, W_self, W_neigh, dH_out, act, need_dH=True, mask=None, rnd=None):
    """Gradients of the SAGE-mean layer.

    dW_self = H^T dZ, dW_neigh = (Abar H)^T dZ,
    dH = dZ W_self^T + Abar^T (dZ W_neigh^T), with Abar^T the stored transpose.
    """
    r = _rnd(rnd)
    H = as_f64(H)
    dZ = _dz(fwd["Z"], dH_out, act, mask)
    out = dict(dZ=dZ, dW_self=r(H).T @ r(dZ), dW_neigh=r(fwd["AH"]).T @ r(dZ))
    if need_dH:
        dP = r(dZ) @ r(W_neigh).T
        if "t_val" in csr:
            agg_t = adjacency(csr, transpose=True) @ dP
        else:
            agg_t = aggregate_transposed(csr, dP)
        out["dH"] = r(dZ) @ r(W_self).T + agg_t
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
