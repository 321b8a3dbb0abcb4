"""One sub-GCN training step and one GIST round (Algorithm 1), in fp64.

A model is a list of per-layer parameters: for GCN layer l a matrix
Theta_l (d_l x d_{l+1}); for GraphSAGE-mean a pair (Theta_self, Theta_neigh)
of that shape.  Hidden layers use ReLU, the last layer the identity, the
loss is mean softmax cross-entropy (Section 3.1: the sub-GCN output has the
global output dimension, so the loss is unchanged).

``sub_gcn_step`` is ``subTrain`` (Section 3.2): forward through eq. (2) on
one mini-batch, loss, backward, one SGD step.  ``gist_round`` is one pass of
the loop body of Algorithm 1: ``subGCNs`` (gather the m slices given the
partitions), zeta local steps per sub-GCN, then ``subAgg``.

``gist_train`` runs the whole of Algorithm 1 (T rounds) with the optimizer
of the paper's experiments, Adam (``oracle.optim``).  The paper does not say
what becomes of Adam's moments at ``subAgg``; two readings are provided:

* ``"carry"``: the moments have the global model's shape and travel with
  the weights -- each round gathers the sub-GCN's slices of Theta, M and V,
  and subAgg writes all three back (entries no sub-GCN owns keep theirs).
  The bias correction counts every local iteration so far, k = t zeta + z + 1.
* ``"reset"``: every round starts each sub-GCN from zero moments, k = z + 1.
"""

import numpy as np

from . import layers as _l
from . import optim as _o


def forward(kind, csr, X, params):
    """Forward pass; returns the list of layer records (AH, Z, H_out) and inputs."""
    H = [_l.as_f64(X)]
    recs = []
    L = len(params)
    for l in range(L):
        act = l < L - 1
        if kind == "gcn":
            rec = _l.gcn_forward(csr, H[-1], params[l], act)
        else:
            rec = _l.sage_forward(csr, H[-1], params[l][0], params[l][1], act)
        recs.append(rec)
        H.append(rec["H_out"])
    return H, recs


def backward(kind, csr, H, recs, params, dlogits):
    """Backward pass from dL/dlogits; returns per-layer gradients and dH records."""
    L = len(params)
    grads = [None] * L
    dHs = [None] * L
    dH = dlogits
    for l in reversed(range(L)):
        act = l < L - 1
        if kind == "gcn":
            b = _l.gcn_backward(csr, H[l], recs[l], params[l], dH, act,
                                need_dH=l > 0)
            grads[l] = b["dW"]
        else:
            b = _l.sage_backward(csr, H[l], recs[l], params[l][0], params[l][1],
                                 dH, act, need_dH=l > 0)
            grads[l] = (b["dW_self"], b["dW_neigh"])
        dH = b.get("dH")
        dHs[l] = dH
    return grads, dHs


def sgd_params(kind, params, grads, lr):
    if kind == "gcn":
        return [_l.sgd(w, g, lr) for w, g in zip(params, grads)]
    return [(_l.sgd(w[0], g[0], lr), _l.sgd(w[1], g[1], lr))
            for w, g in zip(params, grads)]


def sub_gcn_step(kind, csr, X, labels, params, lr):
    """``subTrain``: one SGD step of a sub-GCN on one mini-batch."""
    H, recs = forward(kind, csr, X, params)
    loss, dlogits = _l.softmax_xent(H[-1], labels)
    grads, dHs = backward(kind, csr, H, recs, params, dlogits)
    return dict(loss=loss, H=H, recs=recs, dlogits=dlogits, grads=grads,
                dH=dHs, params=sgd_params(kind, params, grads, lr))


def slice_indices(partitions, L, i):
    """(rows, cols) index lists of sub-GCN i's slice of every layer.

    ``partitions[l]`` is the (idx, offs) partition of hidden width d_l for
    l = 1..L-1 (entries 0 and L unused): the input and output dimensions are
    not partitioned (Section 3.1), so rows of layer 0 and columns of layer
    L-1 are all kept (None).
    """
    out = []
    for l in range(L):
        r = None
        c = None
        if l > 0:
            idx, offs = partitions[l]
            r = list(idx[offs[i]:offs[i + 1]])
        if l + 1 < L:
            idx, offs = partitions[l + 1]
            c = list(idx[offs[i]:offs[i + 1]])
        out.append((r, c))
    return out


def gather_params(kind, theta, sl):
    if kind == "gcn":
        return [_l.gather_slice(theta[l], r, c) for l, (r, c) in enumerate(sl)]
    return [(_l.gather_slice(theta[l][0], r, c), _l.gather_slice(theta[l][1], r, c))
            for l, (r, c) in enumerate(sl)]


def scatter_params(kind, theta, sl, params):
    if kind == "gcn":
        return [_l.subagg(theta[l], r, c, params[l]) for l, (r, c) in enumerate(sl)]
    return [(_l.subagg(theta[l][0], r, c, params[l][0]),
             _l.subagg(theta[l][1], r, c, params[l][1]))
            for l, (r, c) in enumerate(sl)]


def gist_round(kind, theta, partitions, batches, lr, zeta=1):
    """One round of Algorithm 1 on one device, sub-GCNs back to back.

    ``theta``: global parameters; ``partitions[l]``: (idx, offs) of hidden
    width l; ``batches(i, z)`` -> (csr, X, labels) of sub-GCN i's local step
    z.  Returns (new theta, per-sub-GCN trained params, per-step losses).
    """
    L = len(theta)
    m = len(partitions[1][1]) - 1 if L > 1 else 1
    trained, losses = [], []
    for i in range(m):
        sl = slice_indices(partitions, L, i)
        p = gather_params(kind, theta, sl)
        li = []
        for z in range(zeta):
            csr, X, y = batches(i, z)
            st = sub_gcn_step(kind, csr, X, y, p, lr)
            p = st["params"]
            li.append(st["loss"])
        trained.append(p)
        losses.append(li)
    new = theta
    for i in range(m):
        new = scatter_params(kind, new, slice_indices(partitions, L, i), trained[i])
    return new, trained, losses


def zeros_like_params(kind, params):
    if kind == "gcn":
        return [np.zeros(np.shape(w)) for w in params]
    return [(np.zeros(np.shape(a)), np.zeros(np.shape(b))) for a, b in params]


def adam_params(kind, params, grads, M, V, step, lr):
    """Adam on every parameter matrix with its own moments."""
    if kind == "gcn":
        out = [_o.adam(w, g, mm, vv, step, lr) for w, g, mm, vv in zip(params, grads, M, V)]
        return [o[0] for o in out], [o[1] for o in out], [o[2] for o in out]
    P, M1, V1 = [], [], []
    for (ws, wn), (gs, gn), (ms, mn), (vs, vn) in zip(params, grads, M, V):
        a = _o.adam(ws, gs, ms, vs, step, lr)
        b = _o.adam(wn, gn, mn, vn, step, lr)
        P.append((a[0], b[0]))
        M1.append((a[1], b[1]))
        V1.append((a[2], b[2]))
    return P, M1, V1


def sub_gcn_step_adam(kind, csr, X, labels, params, M, V, step, lr):
    """``subTrain`` with Adam: forward, loss, backward, one Adam step."""
    H, recs = forward(kind, csr, X, params)
    loss, dlogits = _l.softmax_xent(H[-1], labels)
    grads, _ = backward(kind, csr, H, recs, params, dlogits)
    P, M1, V1 = adam_params(kind, params, grads, M, V, step, lr)
    return dict(loss=loss, grads=grads, params=P, M=M1, V=V1)


def gist_train(kind, theta, rounds, zeta, lr, partitions, batches, policy="carry"):
    """Algorithm 1 with Adam, sub-GCNs back to back on one device.

    ``partitions(t)`` -> the round's partitions (as for ``slice_indices``);
    ``batches(t, i, z)`` -> (csr, X, labels) of sub-GCN i's local step z.
    Returns (theta, M, V, losses[t][i][z]); M, V are the global moments
    ("carry") or None ("reset").
    """
    if policy not in ("carry", "reset"):
        raise ValueError("policy is 'carry' or 'reset'")
    L = len(theta)
    Mg = zeros_like_params(kind, theta) if policy == "carry" else None
    Vg = zeros_like_params(kind, theta) if policy == "carry" else None
    losses = []
    for t in range(rounds):
        parts = partitions(t)
        m = len(parts[1][1]) - 1 if L > 1 else 1
        trained = []
        lt = []
        for i in range(m):
            sl = slice_indices(parts, L, i)
            p = gather_params(kind, theta, sl)
            if policy == "carry":
                mm, vv = gather_params(kind, Mg, sl), gather_params(kind, Vg, sl)
            else:
                mm, vv = zeros_like_params(kind, p), zeros_like_params(kind, p)
            li = []
            for z in range(zeta):
                csr, X, y = batches(t, i, z)
                k = (t * zeta + z + 1) if policy == "carry" else (z + 1)
                st = sub_gcn_step_adam(kind, csr, X, y, p, mm, vv, k, lr)
                p, mm, vv = st["params"], st["M"], st["V"]
                li.append(st["loss"])
            trained.append((sl, p, mm, vv))
            lt.append(li)
        for sl, p, mm, vv in trained:
            theta = scatter_params(kind, theta, sl, p)
            if policy == "carry":
                Mg = scatter_params(kind, Mg, sl, mm)
                Vg = scatter_params(kind, Vg, sl, vv)
        losses.append(lt)
    return theta, Mg, Vg, losses


def as_float32_params(kind, params):
    if kind == "gcn":
        return [np.asarray(w, dtype=np.float32) for w in params]
    return [(np.asarray(a, dtype=np.float32), np.asarray(b, dtype=np.float32))
            for a, b in params]
