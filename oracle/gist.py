"""One sub-GCN training step and one GIST round (Algorithm 1), in fp64.

A model is a list of per-layer parameters: for GCN layer l a matrix
Theta_l (d_l x d_{l+1}); for GraphSAGE-mean a pair (Theta_self, Theta_neigh)
of that shape; for GAT a triple (Theta_l, a_src, a_dst) with the attention
vectors of length d_{l+1} (``oracle.gat``).  Hidden layers use ReLU, the
last layer the identity, the loss is mean softmax cross-entropy (Section
3.1: the sub-GCN output has the global output dimension, so the loss is
unchanged).

GAT under GIST (Section 2.3: the method applies to GAT unchanged; the paper
trains GAT models with it, Table 2).  A sub-GCN's attention vectors of
layer l are their entries D_{l+1}^(i), the output features its Theta slice
keeps.  The output layer's attention vectors live in the unpartitioned
output dimension, so every sub-GCN trains its own full copy; the paper does
not say how subAgg combines them.  The reading here is that of independent
subnet training, which GIST extends: a parameter that no partition splits
becomes the mean of the m trained copies (for one sub-GCN, the copy itself).
With Adam's "carry" policy its moments are averaged the same way.

``sub_gcn_step`` is ``subTrain`` (Section 2.2): forward through eq. (2) on
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

from . import gat as _g
from . import layers as _l
from . import optim as _o

GAT_SLOPE = 0.2    # LeakyReLU slope of the attention scores (the GAT paper's)


def _parts(kind, p):
    """A layer's parameters as a tuple of arrays."""
    return (p,) if kind == "gcn" else tuple(p)


def _pack(kind, arrs):
    arrs = list(arrs)
    return arrs[0] if kind == "gcn" else tuple(arrs)


def _layer_csr(kind, csr, l):
    """The aggregation matrix of layer l: one matrix for every layer (a
    ``Cluster`` mini-batch), or one per layer (a layer-sampled mini-batch,
    ``oracle.ladies``; GCN only, since its matrices are rectangular)."""
    if isinstance(csr, (list, tuple)):
        if kind != "gcn":
            raise ValueError("per-layer matrices are supported for GCN only")
        return csr[l]
    return csr


def _opt(seq, l):
    return None if seq is None else seq[l]


def forward(kind, csr, X, params, rnd=None, orders=None):
    """Forward pass; returns the list of layer records (AH, Z, H_out) and inputs.

    ``rnd`` rounds the operands of every dense product (the bf16-input
    variant, ``layers.round_bf16``); ``orders[l]`` is GCN layer l's
    association order ("agg" or "xform"; default "agg").  GAT layers take
    neither."""
    H = [_l.as_f64(X)]
    recs = []
    L = len(params)
    if kind == "gat" and rnd is not None:
        raise ValueError("the GAT layers have no rounded variant here")
    for l in range(L):
        act = l < L - 1
        if kind == "gcn":
            rec = _l.gcn_forward(_layer_csr(kind, csr, l), H[-1], params[l], act, rnd=rnd,
                                 order=_opt(orders, l) or "agg")
        elif kind == "gat":
            W, a1, a2 = params[l]
            rec = _g.gat_forward(_layer_csr(kind, csr, l), H[-1], W, a1, a2, act, GAT_SLOPE)
        else:
            rec = _l.sage_forward(_layer_csr(kind, csr, l), H[-1], params[l][0], params[l][1],
                                  act, rnd=rnd)
        recs.append(rec)
        H.append(rec["H_out"])
    return H, recs


def backward(kind, csr, H, recs, params, dlogits, masks=None, pos=None, rnd=None, orders=None):
    """Backward pass from dL/dlogits; returns per-layer gradients and dH records.

    ``masks[l]`` (hidden layers) replaces the ReLU derivative 1[Z_l > 0] and,
    for GAT, ``pos[l]`` the LeakyReLU side of every score of layer l: the
    decisions another evaluation of the same forward took (``layers``).
    ``rnd`` and ``orders`` as in :func:`forward`."""
    L = len(params)
    grads = [None] * L
    dHs = [None] * L
    dH = dlogits
    for l in reversed(range(L)):
        act = l < L - 1
        mask = _opt(masks, l) if act else None
        if kind == "gcn":
            b = _l.gcn_backward(_layer_csr(kind, csr, l), H[l], recs[l], params[l], dH, act,
                                need_dH=l > 0, mask=mask, rnd=rnd,
                                order=_opt(orders, l) or "agg")
            grads[l] = b["dW"]
        elif kind == "gat":
            W, a1, a2 = params[l]
            b = _g.gat_backward(_layer_csr(kind, csr, l), H[l], recs[l], W, a1, a2, dH, act,
                                GAT_SLOPE, need_dH=l > 0, mask=mask, pos=_opt(pos, l))
            grads[l] = (b["dW"], b["da_src"], b["da_dst"])
        else:
            b = _l.sage_backward(_layer_csr(kind, csr, l), H[l], recs[l], params[l][0],
                                 params[l][1], dH, act, need_dH=l > 0, mask=mask, rnd=rnd)
            grads[l] = (b["dW_self"], b["dW_neigh"])
        dH = b.get("dH")
        dHs[l] = dH
    return grads, dHs


def sgd_params(kind, params, grads, lr):
    return [_pack(kind, (_l.sgd(w, g, lr) for w, g in zip(_parts(kind, p), _parts(kind, gr))))
            for p, gr in zip(params, grads)]


def sub_gcn_step(kind, csr, X, labels, params, lr, masks=None, pos=None, rnd=None, orders=None):
    """``subTrain``: one SGD step of a sub-GCN on one mini-batch.

    The optional arguments are those of :func:`forward` and
    :func:`backward`: rounded operands and association orders (the
    bf16-input variant), and the ReLU / LeakyReLU decisions another
    evaluation of the same forward took."""
    H, recs = forward(kind, csr, X, params, rnd=rnd, orders=orders)
    loss, dlogits = _l.softmax_xent(H[-1], labels)
    grads, dHs = backward(kind, csr, H, recs, params, dlogits, masks=masks, pos=pos, rnd=rnd,
                          orders=orders)
    return dict(loss=loss, H=H, recs=recs, dlogits=dlogits, grads=grads,
                dH=dHs, params=sgd_params(kind, params, grads, lr))


def slice_indices(partitions, L, i):
    """(rows, cols) index lists of sub-GCN i's slice of every layer.

    ``partitions[l]`` is the (idx, offs) partition of hidden width d_l for
    l = 1..L-1 (entries 0 and L unused): the input and output dimensions are
    not partitioned (Section 2.1), so rows of layer 0 and columns of layer
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


def _vec_rows(kind):
    """Which parts of a layer are vectors over the output features (GAT's a)."""
    return (False, True, True) if kind == "gat" else (False,) * (1 if kind == "gcn" else 2)


def gather_params(kind, theta, sl):
    """Sub-GCN slices of every layer: rows D_l, columns D_{l+1} of each
    matrix; entries D_{l+1} of each attention vector."""
    out = []
    for l, (r, c) in enumerate(sl):
        arrs = []
        for x, vec in zip(_parts(kind, theta[l]), _vec_rows(kind)):
            arrs.append(_l.gather_slice(x[None, :], None, c)[0] if vec else
                        _l.gather_slice(x, r, c))
        out.append(_pack(kind, arrs))
    return out


def scatter_params(kind, theta, sl, params):
    """Replacement ``subAgg`` of one sub-GCN's slices.  Parts that no
    partition splits (GAT's output-layer attention vectors, c = None) are
    left to :func:`sub_agg`, which averages them."""
    out = []
    for l, (r, c) in enumerate(sl):
        arrs = []
        for x, y, vec in zip(_parts(kind, theta[l]), _parts(kind, params[l]), _vec_rows(kind)):
            if not vec:
                arrs.append(_l.subagg(x, r, c, y))
            elif c is None:
                arrs.append(x)
            else:
                arrs.append(_l.subagg(x[None, :], None, c, y[None, :])[0])
        out.append(_pack(kind, arrs))
    return out


def sub_agg(kind, theta, sls, trained):
    """``subAgg`` of a round: every sub-GCN's slices replace their entries of
    ``theta`` (``sls[i]``, ``trained[i]``); GAT's output-layer attention
    vectors become the mean of the m trained copies."""
    for sl, p in zip(sls, trained):
        theta = scatter_params(kind, theta, sl, p)
    if kind == "gat":
        L = len(theta)
        W = theta[L - 1][0]
        a1 = np.mean([_l.as_f64(p[L - 1][1]) for p in trained], axis=0)
        a2 = np.mean([_l.as_f64(p[L - 1][2]) for p in trained], axis=0)
        theta = list(theta[:L - 1]) + [(W, a1, a2)]
    return theta


def gist_round(kind, theta, partitions, batches, lr, zeta=1, masks=None, steps=None):
    """One round of Algorithm 1 on one device, sub-GCNs back to back.

    ``theta``: global parameters; ``partitions[l]``: (idx, offs) of hidden
    width l; ``batches(i, z)`` -> (csr, X, labels) of sub-GCN i's local step
    z.  Returns (new theta, per-sub-GCN trained params, per-step losses).

    Test use only: ``masks(i, z)``, if given, returns the ReLU decisions
    step z of sub-GCN i takes in its backward (as ``sub_gcn_step``'s
    ``masks``; None keeps its own); ``steps``, if a list, receives every
    local step's result dict in order.
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
            st = sub_gcn_step(kind, csr, X, y, p, lr,
                              masks=None if masks is None else masks(i, z))
            if steps is not None:
                steps.append(st)
            p = st["params"]
            li.append(st["loss"])
        trained.append(p)
        losses.append(li)
    new = sub_agg(kind, theta, [slice_indices(partitions, L, i) for i in range(m)], trained)
    return new, trained, losses


def zeros_like_params(kind, params):
    return [_pack(kind, (np.zeros(np.shape(x)) for x in _parts(kind, p))) for p in params]


def adam_params(kind, params, grads, M, V, step, lr):
    """Adam on every parameter array with its own moments."""
    P, M1, V1 = [], [], []
    for p, g, mm, vv in zip(params, grads, M, V):
        out = [_o.adam(*a, step, lr) for a in zip(_parts(kind, p), _parts(kind, g),
                                                 _parts(kind, mm), _parts(kind, vv))]
        P.append(_pack(kind, (o[0] for o in out)))
        M1.append(_pack(kind, (o[1] for o in out)))
        V1.append(_pack(kind, (o[2] for o in out)))
    return P, M1, V1


def sub_gcn_step_adam(kind, csr, X, labels, params, M, V, step, lr, grad_noise=None,
                      masks=None):
    """``subTrain`` with Adam: forward, loss, backward, one Adam step.

    ``grad_noise`` (test use only, default none): a function applied to
    every gradient array before the Adam step.  A run with a small seeded
    perturbation beside the plain run shows how strongly each element of
    the trained weights depends on its gradients' rounding -- Adam divides
    by the root of the second moment, so elements with small or cancelling
    gradients move by amounts far more sensitive than the gradients
    themselves.  ``masks`` (test use only): the ReLU decisions of the
    backward, as in ``backward``."""
    H, recs = forward(kind, csr, X, params)
    loss, dlogits = _l.softmax_xent(H[-1], labels)
    grads, _ = backward(kind, csr, H, recs, params, dlogits, masks=masks)
    if grad_noise is not None:
        grads = [_pack(kind, (grad_noise(x) for x in _parts(kind, g))) for g in grads]
    P, M1, V1 = adam_params(kind, params, grads, M, V, step, lr)
    return dict(loss=loss, H=H, recs=recs, grads=grads, params=P, M=M1, V=V1)


def gist_train(kind, theta, rounds, zeta, lr, partitions, batches, policy="carry",
               grad_noise=None, masks=None, steps=None):
    """Algorithm 1 with Adam, sub-GCNs back to back on one device.

    ``partitions(t)`` -> the round's partitions (as for ``slice_indices``);
    ``batches(t, i, z)`` -> (csr, X, labels) of sub-GCN i's local step z.
    Returns (theta, M, V, losses[t][i][z]); M, V are the global moments
    ("carry") or None ("reset").  ``grad_noise``: see ``sub_gcn_step_adam``.
    Test use only: ``masks(t, i, z)`` -> the ReLU decisions of that step's
    backward (None keeps its own), ``steps`` (a list) receives every local
    step's result dict in order.
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
                st = sub_gcn_step_adam(kind, csr, X, y, p, mm, vv, k, lr, grad_noise,
                                       masks=None if masks is None else masks(t, i, z))
                if steps is not None:
                    steps.append(st)
                p, mm, vv = st["params"], st["M"], st["V"]
                li.append(st["loss"])
            trained.append((sl, p, mm, vv))
            lt.append(li)
        sls = [tr[0] for tr in trained]
        theta = sub_agg(kind, theta, sls, [tr[1] for tr in trained])
        if policy == "carry":
            Mg = sub_agg(kind, Mg, sls, [tr[2] for tr in trained])
            Vg = sub_agg(kind, Vg, sls, [tr[3] for tr in trained])
        losses.append(lt)
    return theta, Mg, Vg, losses


def as_float32_params(kind, params):
    return [_pack(kind, (np.asarray(x, dtype=np.float32) for x in _parts(kind, p)))
            for p in params]
