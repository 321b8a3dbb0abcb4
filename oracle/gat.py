"""Graph attention layer (GAT) forward and backward in fp64 -- test
infrastructure, never called by the product path.

The paper applies GIST to GAT models (Section 2.3, architecture-agnostic
training; Section 5 and Table 2, Reddit experiments) without restating the
layer; it cites Velickovic et al., "Graph Attention Networks" (ICLR 2018),
whose single-head layer this module follows:

    P = H W                                     (node transform)
    u = P a_src,  v = P a_dst                   (the two halves of a^T [P_i || P_j])
    e_ij = LeakyReLU(u_i + v_j)  for j in N(i) u {i}
    alpha_ij = exp(e_ij) / sum_k exp(e_ik)      (softmax over row i's pattern)
    Z_i = sum_j alpha_ij P_j,   H' = ReLU(Z) for hidden layers, Z for the last.

Readings (the paper is silent): one head; ReLU as the hidden activation,
like the other layers here; LeakyReLU slope given by the caller (0.2 in
the GAT paper); a sub-GCN's slice of a_src and a_dst is their entries
D_{l+1}^(i), the same output features its slice of W keeps (Section 2.1),
so each sub-GCN attends with its own features.

The pattern N(i) u {i} is the stored CSR's (the GCN matrix with self-loops
has exactly that pattern; its values are not used).  The backward is the
chain rule of the forward written out; the softmax row maximum is a
numerical shift and does not change the function.
"""

import numpy as np
import scipy.sparse as sp

from .layers import as_f64, relu


def _edges(csr):
    n = csr["n"]
    rp = np.asarray(csr["rowptr"], dtype=np.int64)
    row = np.repeat(np.arange(n), np.diff(rp))
    col = np.asarray(csr["col"][:rp[-1]], dtype=np.int64)
    return n, rp, row, col


def gat_forward(csr, H, W, a_src, a_dst, act, slope):
    n, rp, row, col = _edges(csr)
    P = as_f64(H) @ as_f64(W)
    u = P @ as_f64(a_src)
    v = P @ as_f64(a_dst)
    pre = u[row] + v[col]
    e = np.where(pre > 0, pre, slope * pre)
    # softmax over each row's entries
    emax = np.full(n, -np.inf)
    np.maximum.at(emax, row, e)
    ex = np.exp(e - emax[row])
    den = np.bincount(row, weights=ex, minlength=n)
    alpha = ex / den[row]
    Aa = sp.csr_matrix((alpha, col, rp), shape=(n, n))
    Z = Aa @ P
    return dict(P=P, u=u, v=v, pre=pre, alpha=alpha, Z=Z, H_out=relu(Z) if act else Z)


def gat_backward(csr, H, fwd, W, a_src, a_dst, dH_out, act, slope, need_dH=True, mask=None,
                 pos=None):
    """Gradients of the GAT layer: dW, da_src, da_dst and (optionally) dH.

    ``mask`` replaces the ReLU derivative 1[Z > 0] and ``pos`` (one bool per
    entry, in the pattern's order) the LeakyReLU side 1[u_i + v_j > 0] of
    each score: the decisions another evaluation of the same forward took
    where a value lies within rounding distance of zero."""
    n, rp, row, col = _edges(csr)
    P, alpha, pre = fwd["P"], fwd["alpha"], fwd["pre"]
    if not act:
        dZ = as_f64(dH_out)
    elif mask is not None:
        dZ = as_f64(dH_out) * np.asarray(mask, dtype=bool)
    else:
        dZ = as_f64(dH_out) * (fwd["Z"] > 0)
    if pos is None:
        pos = pre > 0
    else:
        pos = np.asarray(pos, dtype=bool)
        if pos.shape != pre.shape:
            raise ValueError("pos needs one decision per entry")
    Aa = sp.csr_matrix((alpha, col, rp), shape=(n, n))
    dP = Aa.T @ dZ                                     # through Z = A_alpha P
    dalpha = np.einsum("ek,ek->e", dZ[row], P[col])    # dL/dalpha_ij = dZ_i . P_j
    c = np.bincount(row, weights=alpha * dalpha, minlength=n)
    de = alpha * (dalpha - c[row])                     # softmax backward
    dpre = de * np.where(pos, 1.0, slope)              # LeakyReLU backward
    du = np.bincount(row, weights=dpre, minlength=n)
    dv = np.bincount(col, weights=dpre, minlength=n)
    dP = dP + np.outer(du, as_f64(a_src)) + np.outer(dv, as_f64(a_dst))
    out = dict(dW=as_f64(H).T @ dP, da_src=P.T @ du, da_dst=P.T @ dv, dP=dP, du=du, dv=dv,
               dpre=dpre)
    if need_dH:
        out["dH"] = dP @ as_f64(W).T
    return out
