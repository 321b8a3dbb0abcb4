"""Sub-GCN training step and GIST round, sequenced over the C ABI.

Nothing here computes: each stage is one ``libgist`` call enqueued on the
context's stream (torch only provides the device buffers).

* :class:`SubGCN` -- ``subTrain`` (Section 2.2): layer forward for every
  layer (eq. (2), or the GAT layer), softmax cross-entropy, layer backward
  in reverse, SGD or Adam.
* :class:`GistModel` -- the global model of Algorithm 1 on one device:
  ``subGCNs`` (partition + slice gather), m sub-GCN steps back to back,
  ``subAgg`` (slice scatter), optionally with Adam moments.
* :func:`gist_train` -- Algorithm 1: T rounds of zeta local steps per
  sub-GCN, with SGD or Adam (the optimizer of the paper's experiments).
"""

import numpy as np
import torch

from . import gist as G

GAT_SLOPE = 0.2    # LeakyReLU slope of GAT's attention scores (the GAT paper's)


def _dev(x, device, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(x))
    if dtype is not None:
        t = t.to(dtype)
    return t.to(device, non_blocking=False)


def _wait(event):
    """Wait for a slot's last upload to complete; returns the seconds waited."""
    if event is None:
        return 0.0
    import time
    t0 = time.perf_counter()
    event.synchronize()
    return time.perf_counter() - t0


class DeviceBatch:
    """A mini-batch on the device: CSR (+ transpose for SAGE), features, labels."""

    def __init__(self, csr, X_b, labels_b, device):
        self.n = int(csr["n"])
        self.nnz = int(csr["nnz"])
        self._t = dict(rowptr=_dev(csr["rowptr"], device),
                       col=_dev(csr["col"][:max(self.nnz, 1)], device),
                       val=_dev(csr["val"][:max(self.nnz, 1)], device))
        self.A = G.csr_dev(self.n, self.nnz, self._t["rowptr"], self._t["col"], self._t["val"])
        self.A_T = None
        if "t_rowptr" in csr:
            self._t.update(t_rowptr=_dev(csr["t_rowptr"], device),
                           t_col=_dev(csr["t_col"][:max(self.nnz, 1)], device),
                           t_val=_dev(csr["t_val"][:max(self.nnz, 1)], device))
            self.A_T = G.csr_dev(self.n, self.nnz, self._t["t_rowptr"], self._t["t_col"],
                                 self._t["t_val"])
        self.X = X_b
        self.labels = labels_b

    def rows(self, l):
        """Rows of the activations entering layer l (every layer: the batch)."""
        return self.n

    def adj(self, l):
        return self.A, self.A_T


class BatchSlot:
    """Reusable buffers for one mini-batch: pinned host staging + device copies.

    ``load`` builds the cluster mini-batch CSR on the host directly into
    pinned memory (``gist_build_minibatch_csr``), enqueues asynchronous
    uploads on the current stream, and gathers the batch's feature rows on
    the device (``gist_gather_slice`` with the local->global node map).
    """

    def __init__(self, ctx, norm, cap_n, cap_nnz, d_in, device="cuda", clustered=False):
        self.ctx = ctx
        self.norm = norm
        self.sage = norm == "sage"
        self.clustered = clustered
        self.cap_n, self.cap_nnz = int(cap_n), int(cap_nnz)
        self.device = device
        pin = dict(pin_memory=True)
        i32, f32 = torch.int32, torch.float32
        self.h = dict(rowptr=torch.empty(cap_n + 1, dtype=i32, **pin),
                      col=torch.empty(cap_nnz, dtype=i32, **pin),
                      val=torch.empty(cap_nnz, dtype=f32, **pin),
                      node_map=torch.empty(cap_n, dtype=i32, **pin),
                      labels=torch.empty(cap_n, dtype=i32, **pin))
        if self.sage:
            self.h.update(t_rowptr=torch.empty(cap_n + 1, dtype=i32, **pin),
                          t_col=torch.empty(cap_nnz, dtype=i32, **pin),
                          t_val=torch.empty(cap_nnz, dtype=f32, **pin))
        self.d = {k: torch.empty_like(v, device=device) for k, v in self.h.items()}
        self.X = torch.empty(cap_n, d_in, device=device)
        self.d_in = d_in
        self.uploaded = None
        self.event = None
        self.built = None
        self.sync_s = 0.0

    def build(self, graph_struct, clusters, labels_host):
        """Host half of ``load``: the mini-batch CSR and labels into the pinned
        staging buffers (after the previous upload from them has completed).
        Touches no device memory, so it may run on a worker thread."""
        self.sync_s = _wait(self.uploaded)   # previous upload from the staging buffers done
        q = G.gist_csr()
        q.cap_n, q.cap_nnz = self.cap_n, self.cap_nnz
        h = self.h
        q.rowptr, q.col, q.val = h["rowptr"].data_ptr(), h["col"].data_ptr(), h["val"].data_ptr()
        q.node_map = h["node_map"].data_ptr()
        if self.sage:
            q.t_rowptr, q.t_col, q.t_val = (h["t_rowptr"].data_ptr(), h["t_col"].data_ptr(),
                                            h["t_val"].data_ptr())
        G.build_minibatch_into(graph_struct, clusters, self.norm, q)
        n, nnz = int(q.n), int(q.nnz)
        nm = h["node_map"].numpy()[:n]
        h["labels"].numpy()[:n] = labels_host[nm]
        self.built = (n, nnz)

    def upload(self, X_dev):
        """Device half of ``load``: asynchronous uploads of the built batch and
        the device gather of its feature rows, on the stream of the slot's
        context.  The uploads are kernel pulls from the pinned staging
        buffers (``gist_copy``): they stay on the compute queue, where a
        copy-engine transfer would make the next kernel wait for a hand-off
        between engines."""
        n, nnz = self.built
        h = self.h
        for k in h:
            cnt = n + 1 if k.endswith("rowptr") else (nnz if k.endswith(("col", "val")) else n)
            if cnt:
                G.gist_copy(self.ctx, self.d[k], h[k], 4 * cnt)
        if self.event is None:
            self.event = G.Event()
        G.gist_copy(self.ctx, None, None, 0, self.event)
        self.uploaded = self.event
        Xb = self.X[:n]
        G.gist_gather_slice(self.ctx, X_dev, self.d_in, self.d["node_map"], n, None,
                            self.d_in, Xb, self.d_in)
        return _View(n, nnz, self.d, Xb, self.sage, self.clustered)

    def load(self, graph_struct, clusters, X_dev, labels_host):
        """Build, upload and gather; returns a batch view with n, nnz, A, A_T, X, labels."""
        self.build(graph_struct, clusters, labels_host)
        return self.upload(X_dev)


class FixedBatchSlot:
    """A cluster mini-batch in a fixed layout at the slot's capacities, for
    :class:`ClusterGraphRunner`.

    ``build`` writes the CSR (and the SAGE transpose), node map and labels
    straight into one pinned buffer at fixed offsets and pads them: rows
    past the batch are empty (their row pointers repeat nnz), their node is
    0 and their label 0, and the real row count is stored as one int32 for
    the padded loss.  Shapes are then the same for every batch; empty rows
    aggregate to zero (GCN, SAGE and GAT alike) and the loss ignores them,
    so no result changes.
    """

    _ALIGN = 64

    def __init__(self, ctx, norm, cap_n, cap_nnz, d_in, device="cuda", clustered=False):
        self.ctx, self.d_in, self.device = ctx, d_in, device
        self.clustered = clustered
        self.norm, self.sage = norm, norm == "sage"
        self.cap_n, self.cap_nnz = int(cap_n), int(cap_nnz)
        self.layout = self.fixed_layout(self.sage, self.cap_n, self.cap_nnz)
        self.packed_h = torch.empty(self.layout["total"], dtype=torch.int32, pin_memory=True)
        base = self.packed_h.data_ptr()
        o = self.layout["off"]
        q = G.gist_csr()
        q.cap_n, q.cap_nnz = self.cap_n, self.cap_nnz
        q.rowptr, q.col, q.val = base + 4 * o["rowptr"], base + 4 * o["col"], base + 4 * o["val"]
        q.node_map = base + 4 * o["node_map"]
        if self.sage:
            q.t_rowptr, q.t_col, q.t_val = (base + 4 * o["t_rowptr"], base + 4 * o["t_col"],
                                            base + 4 * o["t_val"])
        self.q = q
        self.event = G.Event()
        self.uploaded = None
        self.n = self.nnz = 0
        self.packed_d = None      # device copy for eager use (upload), made on first use
        self.X = None

    @classmethod
    def fixed_layout(cls, sage, cap_n, cap_nnz):
        pad = lambda n: (int(n) + cls._ALIGN - 1) // cls._ALIGN * cls._ALIGN
        cnt = dict(rowptr=cap_n + 1, col=cap_nnz, val=cap_nnz, node_map=cap_n, labels=cap_n,
                   n_valid=1, coef=3)
        if sage:
            cnt.update(t_rowptr=cap_n + 1, t_col=cap_nnz, t_val=cap_nnz)
        off, o = 0, {}
        for k, c in cnt.items():
            o[k] = off
            off += pad(c)
        return dict(off=o, total=off)

    def build(self, graph_struct, clusters, labels_host, coef=None):
        """Host half: the batch into the fixed layout (after the last upload from
        it); ``coef`` (float32[3], ``gist_adam_coefficients``) rides along for a
        replayed Adam step."""
        self.sync_s = _wait(self.uploaded)
        G.build_minibatch_into(graph_struct, clusters, self.norm, self.q)
        n, nnz = int(self.q.n), int(self.q.nnz)
        h, o, cap = self.packed_h.numpy(), self.layout["off"], self.cap_n
        h[o["rowptr"] + n + 1:o["rowptr"] + cap + 1] = nnz
        if self.sage:
            h[o["t_rowptr"] + n + 1:o["t_rowptr"] + cap + 1] = nnz
        nm = h[o["node_map"]:o["node_map"] + n]
        h[o["labels"]:o["labels"] + n] = labels_host[nm]
        h[o["node_map"] + n:o["node_map"] + cap] = 0
        h[o["labels"] + n:o["labels"] + cap] = 0
        h[o["n_valid"]] = n
        if coef is not None:
            h[o["coef"]:o["coef"] + 3] = np.asarray(coef, dtype=np.float32).view(np.int32)
        self.n, self.nnz = n, nnz

    def upload(self, X_dev):
        """Eager use: copy the batch to this slot's device buffer (one kernel
        pull on the stream of the slot's context) and gather its feature
        rows; returns a view with the real sizes."""
        if self.packed_d is None:
            self.packed_d = torch.empty_like(self.packed_h, device=self.device)
            self.X = torch.empty(self.cap_n, self.d_in, device=self.device)
        c = self.ctx
        G.gist_copy(c, self.packed_d, self.packed_h, 4 * self.layout["total"], self.event)
        self.uploaded = self.event
        o, d, n = self.layout["off"], self.packed_d, self.n
        f32 = torch.float32
        v = dict(rowptr=d[o["rowptr"]:], col=d[o["col"]:],
                 val=d[o["val"]:o["val"] + max(self.nnz, 1)].view(f32),
                 labels=d[o["labels"]:o["labels"] + n])
        if self.sage:
            v.update(t_rowptr=d[o["t_rowptr"]:], t_col=d[o["t_col"]:],
                     t_val=d[o["t_val"]:o["t_val"] + max(self.nnz, 1)].view(f32))
        Xb = self.X[:n]
        if n:
            G.gist_gather_slice(c, X_dev, self.d_in, d[o["node_map"]:], n, None, self.d_in, Xb,
                                self.d_in)
        return _View(n, self.nnz, v, Xb, self.sage, self.clustered)


class BatchPipeline:
    """Mini-batches built ahead of use on host worker threads (cluster
    mini-batches, or LADIES ones with :meth:`ladies`).

    A ring of ``depth`` :class:`BatchSlot` s; batch k is built (host CSR,
    ``gist_build_minibatch_csr`` -- which releases the interpreter lock) into
    slot k mod depth by a pool of ``workers`` threads while earlier batches
    are uploaded and trained on.  ``next()`` returns the batches in the order
    of ``clusters_iter``; each is uploaded on the current stream when it is
    taken, after every kernel enqueued on the slot's previous batch, so a
    slot's device buffers are never overwritten while in use.
    """

    def __init__(self, ctx, norm, cap_n, cap_nnz, d_in, graph_struct, X_dev, labels_host,
                 clusters_iter, depth=8, workers=4, slots=None, build=None):
        from collections import deque
        from concurrent.futures import ThreadPoolExecutor
        self.slots = slots if slots is not None else \
            [BatchSlot(ctx, norm, cap_n, cap_nnz, d_in) for _ in range(depth)]
        self.graph, self.X, self.labels = graph_struct, X_dev, labels_host
        self._build = build if build is not None else \
            (lambda slot, item: slot.build(self.graph, item, self.labels))
        self.src = iter(clusters_iter)
        self.pool = ThreadPoolExecutor(max_workers=workers)
        self.pending = deque()
        self.wait_s = 0.0    # time next() spent waiting for host builds
        self.k = 0           # next batch to submit
        for _ in range(len(self.slots)):
            self._submit()

    @classmethod
    def ladies(cls, ctx, L, b, s, max_degree, d_in, A_handle, X_dev, labels_host, items,
               depth=8, workers=4, fixed=False):
        """A pipeline of LADIES mini-batches; ``items`` yields (output nodes,
        seed[, Adam coefficients]), or a callable returning them (evaluated on
        the worker thread)."""
        slots = [LadiesSlot(ctx, L, b, s, max_degree, d_in, fixed=fixed) for _ in range(depth)]
        def build(slot, item):
            item = item() if callable(item) else item
            slot.build(A_handle, item[0], item[1], labels_host,
                       coef=item[2] if len(item) > 2 else None)
        return cls(ctx, None, 0, 0, d_in, None, X_dev, labels_host, items, workers=workers,
                   slots=slots, build=build)

    def _submit(self):
        try:
            item = next(self.src)
        except StopIteration:
            return
        slot = self.slots[self.k % len(self.slots)]
        self.pending.append((slot, self.pool.submit(self._build, slot, item)))
        self.k += 1

    def take(self, use):
        """Hand the next built slot to ``use(slot)``, which must enqueue every
        read of the slot's host buffers (and record ``slot.uploaded``) before
        it returns; the slot is then refilled with a later batch."""
        slot, fut = self.pending.popleft()
        if not fut.done():           # the host build is behind: time spent waiting for it
            import time
            t0 = time.perf_counter()
            fut.result()
            # less the part of it the build spent waiting for the device to
            # release the slot (back-pressure when the device is the limit)
            self.wait_s += max(0.0, time.perf_counter() - t0 - getattr(slot, "sync_s", 0.0))
        fut.result()
        out = use(slot)
        self._submit()       # reuses this slot: its build waits for the upload just enqueued
        return out

    def take_many(self, n, use):
        """Hand the next ``n`` built slots to ``use(slots)`` together, with the
        contract of :meth:`take` for each of them; then refill them."""
        import time
        items = [self.pending.popleft() for _ in range(n)]
        for slot, fut in items:
            if not fut.done():
                t0 = time.perf_counter()
                fut.result()
                self.wait_s += max(0.0, time.perf_counter() - t0 - getattr(slot, "sync_s", 0.0))
            fut.result()
        out = use([slot for slot, _ in items])
        for _ in range(n):
            self._submit()
        return out

    def next(self):
        """The next batch, uploaded on the current stream."""
        return self.take(lambda slot: slot.upload(self.X))

    def close(self):
        for _, fut in self.pending:
            fut.cancel()
        self.pool.shutdown(wait=True)


class _View:
    def __init__(self, n, nnz, d, X, sage, clustered=False):
        self.n, self.nnz = n, nnz
        self.clustered = clustered   # a cluster mini-batch: GIST_LAYER_CLUSTERED applies
        self.A = G.csr_dev(n, nnz, d["rowptr"], d["col"], d["val"])
        self.A_T = G.csr_dev(n, nnz, d["t_rowptr"], d["t_col"], d["t_val"]) if sage else None
        self.X = X
        self.labels = d["labels"][:n]

    def rows(self, l):
        return self.n

    def adj(self, l):
        return self.A, self.A_T


class LadiesSlot:
    """Reusable buffers for one LADIES mini-batch (Section 5.4, Appendix A.6:
    layer-wise sampling in place of graph partitioning, GCN only).

    ``build`` runs ``gist_ladies_sample`` on the host into pinned per-layer
    staging arrays sized by the capacities, then packs what it produced
    (every layer's node list, row pointers, entries and transpose, and the
    output nodes' labels) into one pinned transfer buffer; ``upload``
    enqueues that buffer as a single copy on the current stream and gathers
    the input layer's feature rows (V_0) on the device.  Capacities follow
    from the batch size b and the draws s per layer: |V_l| <= b + (L - l) s,
    and a layer's entries are at most its rows times (largest degree + 1).

    With ``fixed=True`` the transfer buffer has a fixed layout at the
    capacities (see :meth:`fixed_layout`), every node set padded to its
    capacity: padded rows are empty (their row pointers repeat the last
    one), padded input nodes are node 0.  The layer shapes are then the
    same for every batch, which :class:`LadiesGraphRunner` relies on; the
    results are those of the unpadded batch, since empty rows aggregate to
    zero and contribute nothing to any gradient.
    """

    _ORDER = ("nodes", "rowptr", "t_rowptr", "col", "t_col", "val", "t_val")
    _ALIGN = 64      # elements (256 bytes) between packed arrays

    def __init__(self, ctx, L, b, s, max_degree, d_in, device="cuda", fixed=False,
                 fixed_nnz_per_row=16):
        self.ctx, self.L, self.b, self.s = ctx, L, int(b), int(s)
        self.device = device
        self.fixed = fixed
        pin = dict(pin_memory=True)
        i32, f32 = torch.int32, torch.float32
        self.caps = []
        for l in range(L):
            cap_n = self.b + (L - l) * self.s
            rows = self.b + (L - l - 1) * self.s
            self.caps.append((cap_n, rows * (int(max_degree) + 1)))
        self.h = []
        self.arr = (G.gist_ladies_layer * L)()
        total = 0
        for l, (cn, cz) in enumerate(self.caps):
            h = dict(nodes=torch.empty(cn, dtype=i32, **pin),
                     rowptr=torch.empty(cn + 1, dtype=i32, **pin),
                     col=torch.empty(cz, dtype=i32, **pin), val=torch.empty(cz, dtype=f32, **pin),
                     t_rowptr=torch.empty(cn + 1, dtype=i32, **pin),
                     t_col=torch.empty(cz, dtype=i32, **pin),
                     t_val=torch.empty(cz, dtype=f32, **pin))
            self.h.append(h)
            a = self.arr[l]
            a.cap_n, a.cap_nnz = cn, cz
            for k, v in h.items():
                setattr(a, k, v.data_ptr())
                total += self._pad(v.numel())
        total += self._pad(self.b)          # labels
        if fixed:
            self.layout = self.fixed_layout(L, b, s, fixed_nnz_per_row)
            total = max(total, self.layout["total"])
        # transfer buffer: 4-byte elements (int32, float32 viewed as int32)
        self.packed_h = torch.empty(total, dtype=i32, **pin)
        self.packed_d = torch.empty(total, dtype=i32, device=device)
        if fixed:
            # the sampler writes straight into the fixed layout's sections
            self.arr_fixed = (G.gist_ladies_layer * L)()
            base = self.packed_h.data_ptr()
            for l, fl in enumerate(self.layout["layers"]):
                a = self.arr_fixed[l]
                a.cap_n, a.cap_nnz = fl["n_in"], fl["nnz"]
                for k in self._ORDER:
                    setattr(a, k, base + 4 * fl["off"][k])
        self.X = torch.empty(self.caps[0][0], d_in, device=device)
        self.d_in = d_in
        self.event = G.Event()      # recorded by gist_replay_launch after its copy
        self.uploaded = None
        self.built = None

    @classmethod
    def _pad(cls, n):
        return (int(n) + cls._ALIGN - 1) // cls._ALIGN * cls._ALIGN

    @classmethod
    def fixed_layout(cls, L, b, s, nnz_per_row):
        """Offsets of the fixed transfer layout: per layer l the padded sizes
        (rows |V_{l+1}| cap, input nodes |V_l| cap, entries cap) and each
        array's offset, then the labels; ``total`` elements in all.  Both row
        pointer arrays hold |V_l| cap + 1 entries, the sampler's capacity
        contract."""
        off, layers = 0, []
        for l in range(L):
            n_in = b + (L - l) * s
            n_out = b + (L - l - 1) * s
            nnz = n_out * int(nnz_per_row)
            cnt = dict(nodes=n_in, rowptr=n_in + 1, t_rowptr=n_in + 1, col=nnz, t_col=nnz,
                       val=nnz, t_val=nnz)
            o = {}
            for k in cls._ORDER:
                o[k] = off
                off += cls._pad(cnt[k])
            layers.append(dict(n_out=n_out, n_in=n_in, nnz=nnz, off=o))
        lab = off
        off += cls._pad(b)
        coef = off
        off += cls._pad(3)
        return dict(layers=layers, labels=lab, coef=coef, total=off)

    def build(self, A_handle, batch, seed, labels_host, coef=None):
        """Host half: sample the layers, pack them and the output nodes' labels
        (and, fixed layout, the Adam coefficients ``coef`` of a replayed step)."""
        self.sync_s = _wait(self.uploaded)   # the previous upload from packed_h is done
        batch = np.asarray(batch, dtype=np.int32)
        nb = batch.shape[0]
        if nb > self.b or (self.fixed and nb != self.b):
            raise ValueError("batch size does not match the slot")
        packed = self.packed_h.numpy()
        if self.fixed:
            try:
                G.ladies_sample_into(A_handle, batch, self.L, self.s, seed, self.arr_fixed)
            except G.GistError as e:   # more entries than the fixed layout holds
                if e.status != G.GIST_E_NOMEM:
                    raise
            else:
                sizes, offs = [], []
                for l, fl in enumerate(self.layout["layers"]):
                    a = self.arr_fixed[l]
                    n_out, n_in, nnz = int(a.n_out), int(a.n_in), int(a.nnz)
                    o = fl["off"]    # pad to the fixed shapes: empty rows, node 0
                    packed[o["rowptr"] + n_out + 1:o["rowptr"] + fl["n_out"] + 1] = nnz
                    packed[o["t_rowptr"] + n_in + 1:o["t_rowptr"] + fl["n_in"] + 1] = nnz
                    packed[o["nodes"] + n_in:o["nodes"] + fl["n_in"]] = 0
                    offs.append(o)
                    sizes.append((n_out, n_in, nnz))
                lab = self.layout["labels"]
                packed[lab:lab + nb] = labels_host[batch]
                if coef is not None:
                    c = self.layout["coef"]
                    packed[c:c + 3] = np.asarray(coef, dtype=np.float32).view(np.int32)
                self.built = (nb, sizes, offs, lab, self.layout["total"], True)
                return
        # compact layout: sample into the staging arrays, pack what was produced
        G.ladies_sample_into(A_handle, batch, self.L, self.s, seed, self.arr)
        off, offs, sizes = 0, [], []
        for l in range(self.L):
            a = self.arr[l]
            n_out, n_in, nnz = int(a.n_out), int(a.n_in), int(a.nnz)
            cnt = dict(nodes=n_in, rowptr=n_out + 1, t_rowptr=n_in + 1)
            o = {}
            for k in self._ORDER:
                c = cnt.get(k, nnz)
                o[k] = off
                off += self._pad(c)
                packed[o[k]:o[k] + c] = self.h[l][k].numpy()[:c].view(np.int32)
            offs.append(o)
            sizes.append((n_out, n_in, nnz))
        packed[off:off + nb] = labels_host[batch]
        self.built = (nb, sizes, offs, off, off + self._pad(nb), False)

    def fits_fixed(self):
        """Whether the last built batch is in the fixed layout (else it is
        packed compactly: its entries exceeded the fixed capacity)."""
        return self.built[5]

    def upload(self, X_dev):
        """Device half: one asynchronous copy on the current stream and the
        gather of the input nodes' features."""
        nb, sizes, offs, lab, total, fits = self.built
        d = self.packed_d
        G.gist_copy(self.ctx, d, self.packed_h, 4 * total, self.event)
        self.uploaded = self.event
        f32 = torch.float32
        views = []
        for l, (n_out, n_in, nnz) in enumerate(sizes):
            o = offs[l]
            v = {k: d[o[k]:] for k in ("nodes", "rowptr", "t_rowptr", "col", "t_col")}
            v["val"] = d[o["val"]:o["val"] + max(nnz, 1)].view(f32)
            v["t_val"] = d[o["t_val"]:o["t_val"] + max(nnz, 1)].view(f32)
            views.append(v)
        n0 = sizes[0][1]
        Xb = self.X[:n0]
        if n0:
            G.gist_gather_slice(self.ctx, X_dev, self.d_in, views[0]["nodes"], n0, None,
                                self.d_in, Xb, self.d_in)
        return LadiesView(sizes, views, Xb, d[lab:lab + nb])

    def load(self, A_handle, batch, seed, X_dev, labels_host):
        self.build(A_handle, batch, seed, labels_host)
        return self.upload(X_dev)


class _Replayer:
    """Shared part of the replay runners: a side-stream context to record
    on, and one recorded step per (parameter set, optimizer state, lr).

    A step is recorded with SGD (its learning rate fixed in the recording),
    or with Adam (``adam`` = (M, V) moment slices): then the coefficients
    are read from the batch's device buffer (``gist_adam_update_dev``), so
    the same recording serves every step k and both moment policies.
    """

    def _init_replay(self, ctx):
        self.ctx = ctx
        self.cap_stream = torch.cuda.Stream()
        self.cap_ctx = G.Context(ctx.device, stream=self.cap_stream.cuda_stream)
        self.replays = {}

    def _backward_update(self, view, params, lr, adam):
        """The recorded backward pass and update: SGD fused into the backward
        pass, or Adam with the batch's coefficients."""
        if adam is None:
            self.run.backward(view, params, sgd_lr=lr)
        else:
            self.run.backward(view, params)
            M, V = adam
            self.run.adam_dev(params, M, V, self.coef_dev)

    def _capture(self, params, lr, adam):
        torch.cuda.synchronize()    # everything the recording reads exists and is written
        G.gist_capture_begin(self.cap_ctx)
        try:
            self._body(params, lr, adam)
        finally:
            replay = G.gist_capture_end(self.cap_ctx)
        return replay

    def _replay(self, slot, params, lr, adam):
        key = (tuple(p.data_ptr() for p in params),
               None if adam is None else tuple(t.data_ptr() for m in adam for t in m),
               None if adam is not None else float(lr))
        r = self.replays.get(key)
        if r is None:
            r = self.replays[key] = self._capture(params, lr, adam)
        G.gist_replay_launch(self.ctx, r, self.dev, slot.packed_h, self.nbytes, slot.event)
        slot.uploaded = slot.event

    @property
    def graphs(self):
        return self.replays

    @property
    def loss(self):
        return self.run.loss


class ClusterGraphRunner(_Replayer):
    """Sub-GCN steps on cluster mini-batches replayed from HIP graphs (the
    counterpart of :class:`LadiesGraphRunner` for GCN, SAGE and GAT layers).

    Every batch is run at the capacity shape of :class:`FixedBatchSlot` (n
    rows, nnz entries): the step (feature gather, forward, padded loss,
    backward, SGD or Adam) is recorded once per parameter set on a
    side-stream context, and each step is one ``gist_replay_launch`` that
    pulls the batch from pinned memory into this runner's buffer.
    """

    def __init__(self, ctx, kind, widths, cap_n, cap_nnz, d_in, X_dev, dtype=G.GIST_DTYPE_F32,
                 device="cuda", clustered=False):
        self._init_replay(ctx)
        self.d_in, self.X_dev = d_in, X_dev
        norm = "sage" if kind == "sage" else "gcn"
        self.layout = FixedBatchSlot.fixed_layout(norm == "sage", cap_n, cap_nnz)
        self.dev = torch.empty(self.layout["total"], dtype=torch.int32, device=device)
        o, d = self.layout["off"], self.dev
        f32 = torch.float32
        view = dict(rowptr=d[o["rowptr"]:], col=d[o["col"]:],
                    val=d[o["val"]:o["val"] + cap_nnz].view(f32),
                    labels=d[o["labels"]:o["labels"] + cap_n])
        if norm == "sage":
            view.update(t_rowptr=d[o["t_rowptr"]:], t_col=d[o["t_col"]:],
                        t_val=d[o["t_val"]:o["t_val"] + cap_nnz].view(f32))
        self.node_map = d[o["node_map"]:o["node_map"] + cap_n]
        self.coef_dev = d[o["coef"]:o["coef"] + 3].view(f32)
        self.X = torch.empty(cap_n, d_in, device=device)
        self.view = _View(cap_n, cap_nnz, view, self.X, norm == "sage", clustered)
        self.view.n_dev = d[o["n_valid"]:o["n_valid"] + 1]
        self.cap_n = cap_n
        self.run = SubGCN(self.cap_ctx, kind, widths, cap_n, dtype=dtype, device=device)
        self.run.prepare(self.view)
        self.nbytes = 4 * self.layout["total"]

    def _body(self, params, lr, adam):
        G.gist_gather_slice(self.cap_ctx, self.X_dev, self.d_in, self.node_map, self.cap_n, None,
                            self.d_in, self.X, self.d_in)
        self.run.forward(self.view, params)
        self.run.loss_and_grad(self.view)
        self._backward_update(self.view, params, lr, adam)

    def step(self, slot, params, lr, adam=None):
        """One sub-GCN step on the batch built in ``slot``; ``adam`` = (M, V)
        for Adam with the coefficients the slot carries."""
        self._replay(slot, params, lr, adam)


class LadiesGraphRunner(_Replayer):
    """Sub-GCN steps on LADIES mini-batches replayed from HIP graphs.

    A LADIES step is a few dozen small launches (c7: GEMMs of at most
    1536 x 602 x 64), so issuing them one by one costs more host time than
    they take on the device.  Here each step is recorded once
    (``gist_capture_begin`` / ``_end`` on a context of its own, on a side
    stream) at the fixed shapes of ``LadiesSlot(fixed=True)``: the feature
    gather, every layer's forward, the loss, every layer's backward and the
    update.  Per step the host then makes one library call,
    ``gist_replay_launch``: the copy of the batch into this runner's device
    buffer, an event that frees the slot, and the replay, on the stream of
    ``ctx``.
    """

    def __init__(self, ctx, widths, L, b, s, d_in, X_dev, dtype=G.GIST_DTYPE_F32,
                 fixed_nnz_per_row=16, device="cuda"):
        self._init_replay(ctx)
        self.L, self.d_in, self.X_dev = L, d_in, X_dev
        self.layout = LadiesSlot.fixed_layout(L, b, s, fixed_nnz_per_row)
        self.dev = torch.empty(self.layout["total"], dtype=torch.int32, device=device)
        lay = self.layout["layers"]
        sizes = [(fl["n_out"], fl["n_in"], fl["nnz"]) for fl in lay]
        views = []
        for fl in lay:
            o = fl["off"]
            v = {k: self.dev[o[k]:] for k in ("nodes", "rowptr", "t_rowptr", "col", "t_col")}
            v["val"] = self.dev[o["val"]:o["val"] + fl["nnz"]].view(torch.float32)
            v["t_val"] = self.dev[o["t_val"]:o["t_val"] + fl["nnz"]].view(torch.float32)
            views.append(v)
        self.n0 = lay[0]["n_in"]
        self.X = torch.empty(self.n0, d_in, device=device)
        lab, c = self.layout["labels"], self.layout["coef"]
        self.view = LadiesView(sizes, views, self.X, self.dev[lab:lab + b])
        self.coef_dev = self.dev[c:c + 3].view(torch.float32)
        self.nodes0 = views[0]["nodes"]
        self.run = SubGCN(self.cap_ctx, "gcn", widths, self.n0, dtype=dtype, device=device)
        self.run.prepare(self.view)
        self.nbytes = 4 * self.layout["total"]

    def _body(self, params, lr, adam):
        G.gist_gather_slice(self.cap_ctx, self.X_dev, self.d_in, self.nodes0, self.n0, None,
                            self.d_in, self.X, self.d_in)
        self.run.forward(self.view, params)
        self.run.loss_and_grad(self.view)
        self._backward_update(self.view, params, lr, adam)

    def step(self, slot, params, lr, adam=None):
        """One sub-GCN step on the batch built in ``slot`` (fixed layout): one
        library call copies it into this runner's buffer and replays the step
        (recorded on first use of these parameters).  ``adam`` = (M, V) for
        Adam with the coefficients the slot carries."""
        if not slot.fits_fixed():    # rare: too many entries for the fixed layout
            if adam is not None:
                raise ValueError("a batch beyond the fixed layout cannot take a replayed "
                                 "Adam step")
            self.cap_ctx.set_stream(torch.cuda.current_stream().cuda_stream)
            try:
                self.run.step(slot.upload(self.X_dev), params, lr)
            finally:
                self.cap_ctx.set_stream(self.cap_stream.cuda_stream)
            return
        self._replay(slot, params, lr, adam)


class RoundReplayer:
    """Whole GIST rounds replayed from HIP graphs: the fused subAgg + gather
    of :meth:`GistModel.begin_round` and the m sub-GCN steps (each: the copy of
    its mini-batch from pinned memory, the step recorded by ``runner``, SGD
    fused into the backward pass) recorded as one graph, so that a round
    costs the host one partition upload and one launch instead of a few
    library calls per sub-GCN.

    One recording per state the round starts from: the model's partition
    slot, slice buffer and pending subAgg, and the pipeline slots that hold
    the round's m mini-batches (with a ring of 4m slots the state repeats
    every four rounds, so after the first five rounds every round is a
    replay).  SGD, one local step per sub-GCN, one stream.  A round with a
    mini-batch beyond the runner's fixed layout runs step by step instead.
    """

    def __init__(self, model, runner, pipe, lr):
        if not model.fused or model.adam is not None:
            raise ValueError("round replays need the fused subAgg and SGD")
        self.model, self.runner, self.pipe, self.lr = model, runner, pipe, float(lr)
        self.replays = {}
        self.event = G.Event()
        self.stepwise_rounds = 0

    def _capture(self, slots):
        m, run = self.model, self.runner
        torch.cuda.synchronize()    # everything the recording reads exists and is written
        ctx0 = m.ctx
        m.ctx = run.cap_ctx
        G.gist_capture_begin(run.cap_ctx)
        try:
            m._begin_state(m._begin_launches())
            for i, slot in enumerate(slots):
                G.gist_copy(run.cap_ctx, run.dev, slot.packed_h, run.nbytes)
                run._body(m.params[i], self.lr, None)
        finally:
            replay = G.gist_capture_end(run.cap_ctx)
            m.ctx = ctx0
        return replay

    def _round(self, slots):
        m, run = self.model, self.runner
        if not all(getattr(s, "fits_fixed", lambda: True)() for s in slots):
            self.stepwise_rounds += 1
            m.begin_round()
            for i, slot in enumerate(slots):
                run.step(slot, m.params[i], self.lr)
            return
        key = (m._slot, m.buf, m.pending, tuple(s.packed_h.data_ptr() for s in slots))
        r = self.replays.get(key)
        if r is None:
            r = self.replays[key] = self._capture(slots)
        else:
            m._begin_state(1 - m.buf if m.pending is not None else m.buf)
        G.gist_replay_launch(run.ctx, r)
        G.gist_copy(run.ctx, None, None, 0, self.event)   # the slots' batches are read
        for slot in slots:
            slot.uploaded = self.event

    def round(self, seeds):
        """One round: ``subGCNs`` with the partition seeds ``seeds`` ({l: seed}),
        the replayed round, and the (deferred) subAgg bookkeeping."""
        self.model.set_partitions(seeds)
        self.pipe.take_many(self.model.m, self._round)
        self.model.end_round()


class LadiesView:
    """A loaded LADIES mini-batch: per-layer rectangular matrices (rows
    V_{l+1}, columns V_l) with their transposes, the features of V_0 and
    the labels of the output nodes V_L."""

    def __init__(self, sizes, d, X, labels):
        self.sizes = sizes
        self._rows = [s[1] for s in sizes] + [sizes[-1][0]]
        self._A = [G.csr_dev(n_out, nnz, d[l]["rowptr"], d[l]["col"], d[l]["val"])
                   for l, (n_out, n_in, nnz) in enumerate(sizes)]
        self._AT = [G.csr_dev(n_in, nnz, d[l]["t_rowptr"], d[l]["t_col"], d[l]["t_val"])
                    for l, (n_out, n_in, nnz) in enumerate(sizes)]
        self.X = X
        self.labels = labels
        self.n = self._rows[-1]
        self.nnz = sum(s[2] for s in sizes)

    def rows(self, l):
        """|V_l|: rows of the activations entering layer l (l = L: the output nodes)."""
        return self._rows[l]

    def adj(self, l):
        return self._A[l], self._AT[l]


def relu_chain_flags(l, L):
    """Backward flags of layer l of L that fuse every hidden layer's ReLU
    derivative into the kernel writing the gradient it multiplies: a hidden
    layer's dH_out arrives as dZ (GIST_LAYER_DZ_IN), and every layer above the
    first writes dH times the layer below's derivative (GIST_LAYER_MASK_DH).
    No separate ReLU-derivative pass runs; the results are bitwise the same."""
    return (G.GIST_LAYER_DZ_IN if l < L - 1 else 0) | (G.GIST_LAYER_MASK_DH if l > 0 else 0)


class SubGCN:
    """Buffers and call sequence of one sub-GCN's training step.

    ``widths`` are the slice widths s_0..s_L; ``kind`` is "gcn", "sage" or
    "gat".  Parameters are device tensors ``params[l]`` of shape
    (s_l, s_{l+1}) (SAGE: (2 s_l, s_{l+1}), W_self stacked over W_neigh;
    GAT: (s_l + 2, s_{l+1}), Theta followed by the rows a_src and a_dst), and
    the gradients ``dW[l]`` have the same layout, so one optimizer call
    updates a layer.  A GAT batch's CSR is the pattern of A + I (the GCN
    matrix; its values are not read).
    """

    def __init__(self, ctx, kind, widths, n_cap, dtype=G.GIST_DTYPE_F32, device="cuda",
                 order=G.GIST_ORDER_AUTO):
        if kind not in ("gcn", "sage", "gat"):
            raise ValueError("kind is 'gcn', 'sage' or 'gat'")
        self.ctx = ctx
        self.kind = kind
        self.gat = kind == "gat"
        self.nnz_cap = 0
        self.alpha = None
        self.widths = list(widths)
        self.L = len(widths) - 1
        self.dtype = dtype
        self.order = order
        self.device = device
        self.lkind = G.GIST_LAYER_SAGE_MEAN if kind == "sage" else G.GIST_LAYER_GCN
        self.n_cap = 0
        self.ws = torch.empty(0, dtype=torch.uint8, device=device)
        self._alloc(n_cap)
        self.dW = [torch.empty(self.wrows(l), widths[l + 1], device=device)
                   for l in range(self.L)]
        self.loss = torch.zeros(1, device=device)

    def wrows(self, l):
        if self.gat:
            return self.widths[l] + 2
        return (2 if self.kind == "sage" else 1) * self.widths[l]

    def _alloc(self, n_cap):
        w, d = self.widths, self.device
        self.n_cap = n_cap
        self.H = [None] + [torch.empty(n_cap, w[l + 1], device=d) for l in range(self.L)]
        # GCN / SAGE save the aggregation Abar H; GAT saves the transform P = H Theta
        self.agg = [torch.empty(n_cap, w[l + 1] if self.gat else w[l], device=d)
                    for l in range(self.L)]
        # dH[l]: the gradient reaching H_l; for GCN / SAGE times its ReLU
        # derivative 1[H_l > 0], which the layer above applies (MASK_DH)
        self.dH = [torch.empty(n_cap, w[l], device=d) for l in range(self.L)]
        self.dlogits = torch.empty(n_cap, w[self.L], device=d)
        self.loss_ws = torch.empty(G.gist_softmax_xent_workspace(n_cap), dtype=torch.uint8,
                                   device=d)

    def desc(self, l, n, nnz=0, n_in=0, clustered=False):
        """Layer l's descriptor for n output rows (n_in input rows, 0: n);
        ``clustered``: the batch is a cluster mini-batch (GIST_LAYER_CLUSTERED)."""
        act = G.GIST_ACT_RELU if l < self.L - 1 else G.GIST_ACT_NONE
        if self.gat:
            return G.gat_desc(n, nnz, self.widths[l], self.widths[l + 1], act, self.dtype,
                              GAT_SLOPE)
        return G.layer_desc(self.lkind, act, n, self.widths[l], self.widths[l + 1],
                            self.dtype, self.order, n_in=n_in,
                            flags=G.GIST_LAYER_CLUSTERED if clustered else 0)

    def _ldesc(self, batch, l):
        return self.desc(l, batch.rows(l + 1), batch.nnz, batch.rows(l),
                         getattr(batch, "clustered", False))

    def _workspace(self, batch):
        need = 0
        for l in range(self.L):
            if self.gat:
                f, b = G.gist_gat_workspace_size(self._ldesc(batch, l))
            else:
                f, b = G.gist_layer_workspace_size(self._ldesc(batch, l))
            need = max(need, f, b)
        if self.ws.numel() < need:
            self.ws = torch.empty(need, dtype=torch.uint8, device=self.device)
        return self.ws

    def _gat_parts(self, t, l):
        """(Theta, a_src, a_dst) views of a GAT layer's stacked parameters."""
        s = self.widths[l]
        return t[:s], t[s], t[s + 1]

    def forward(self, batch, params):
        """Every layer's forward.  A batch gives the rows entering each layer
        (``rows(l)``) and each layer's matrix (``adj(l)``): the same for every
        layer for a cluster mini-batch, per layer for a LADIES one."""
        nnz = batch.nnz
        n_max = max(batch.rows(l) for l in range(self.L + 1))
        if n_max > self.n_cap:
            self._alloc(n_max)
        if self.gat and (self.alpha is None or nnz > self.nnz_cap):
            self.nnz_cap = max(nnz, 1)
            self.alpha = [torch.empty(self.nnz_cap, device=self.device) for _ in range(self.L)]
        ws = self._workspace(batch)
        H = batch.X
        for l in range(self.L):
            n = batch.rows(l + 1)
            A = batch.adj(l)[0]
            out = self.H[l + 1][:n]
            if self.gat:
                W, a1, a2 = self._gat_parts(params[l], l)
                G.gist_gat_layer_fwd(self.ctx, self._ldesc(batch, l), A, H, W, a1, a2,
                                     self.agg[l][:n], self.alpha[l][:nnz], out, ws)
            else:
                G.gist_gcn_layer_fwd(self.ctx, self._ldesc(batch, l), A, H, params[l],
                                     self.agg[l][:n], out, ws)
            H = out
        return self.H[self.L][:batch.rows(self.L)]

    def loss_and_grad(self, batch, loss_out=None):
        """Loss into ``loss_out`` (a one-element device tensor) or ``self.loss``.
        A padded batch (``n_dev``: its real row count on the device) takes the
        mean over its real rows."""
        n = batch.rows(self.L)
        out = self.loss if loss_out is None else loss_out
        n_dev = getattr(batch, "n_dev", None)
        if n_dev is not None:
            G.gist_softmax_xent_padded(self.ctx, n, self.widths[-1], self.H[self.L][:n],
                                       batch.labels, n_dev, out, self.dlogits[:n], self.loss_ws)
        else:
            G.gist_softmax_xent(self.ctx, n, self.widths[-1], self.H[self.L][:n], batch.labels,
                                out, self.dlogits[:n], self.loss_ws)

    def prepare(self, batch):
        """Allocate every buffer a step on ``batch`` needs (before a capture)."""
        n_max = max(batch.rows(l) for l in range(self.L + 1))
        if n_max > self.n_cap:
            self._alloc(n_max)
        if self.gat and (self.alpha is None or batch.nnz > self.nnz_cap):
            self.nnz_cap = max(batch.nnz, 1)
            self.alpha = [torch.empty(self.nnz_cap, device=self.device) for _ in range(self.L)]
        self._workspace(batch)

    def backward(self, batch, params, sgd_lr=None):
        """Every layer's backward pass into ``self.dW``; with ``sgd_lr`` also
        the SGD step.  A GCN / SAGE layer takes it inside its backward pass
        (``gist_gcn_layer_bwd_sgd``: the weight-gradient GEMM updates the
        slice in place, after the input gradient has read it; no dW); GAT
        layers after the pass (``gist_sgd_update``)."""
        fused = sgd_lr is not None and not self.gat
        nnz = batch.nnz
        ws = self._workspace(batch)
        dout = self.dlogits[:batch.rows(self.L)]
        prev_A = None
        for l in reversed(range(self.L)):
            n, n_in = batch.rows(l + 1), batch.rows(l)
            A, A_T = batch.adj(l)
            Hin = batch.X if l == 0 else self.H[l][:n_in]
            dH = self.dH[l][:n_in] if l > 0 else None
            if self.gat:
                W, a1, a2 = self._gat_parts(params[l], l)
                gW, g1, g2 = self._gat_parts(self.dW[l], l)
                desc = self._ldesc(batch, l)
                if A is prev_A:   # same pattern: the layer above left its mirror map in ws
                    desc.flags = G.GIST_GAT_MIRROR_IN_WS
                prev_A = A
                G.gist_gat_layer_bwd(self.ctx, desc, A, Hin,
                                     self.agg[l][:n], self.alpha[l][:nnz], self.H[l + 1][:n],
                                     W, a1, a2, dout, gW, g1, g2, dH, ws)
            elif fused:
                desc = self._ldesc(batch, l)
                desc.flags |= relu_chain_flags(l, self.L)
                G.gist_gcn_layer_bwd_sgd(self.ctx, desc, A, A_T, Hin,
                                         self.agg[l][:n], self.H[l + 1][:n], params[l], dout,
                                         sgd_lr, dH, ws)
            else:
                desc = self._ldesc(batch, l)
                desc.flags |= relu_chain_flags(l, self.L)
                G.gist_gcn_layer_bwd(self.ctx, desc, A, A_T, Hin,
                                     self.agg[l][:n], self.H[l + 1][:n], params[l], dout,
                                     self.dW[l], dH, ws)
            dout = dH
        if sgd_lr is not None and not fused:
            self.sgd(params, sgd_lr)

    def sgd(self, params, lr):
        for l in range(self.L):
            G.gist_sgd_update(self.ctx, params[l], self.dW[l], params[l].numel(), lr)

    def adam(self, params, M, V, lr, step, fresh=False, betas=(0.9, 0.999), eps=1e-8):
        """Adam on every layer's slice with its moments M[l], V[l]; ``fresh``
        restarts the moments from zero (gist_adam_update's GIST_ADAM_FRESH)."""
        flags = G.GIST_ADAM_FRESH if fresh else 0
        for l in range(self.L):
            G.gist_adam_update(self.ctx, params[l], self.dW[l], M[l], V[l], params[l].numel(),
                               lr, step, betas[0], betas[1], eps, flags)

    def adam_dev(self, params, M, V, coef_dev, betas=(0.9, 0.999), eps=1e-8):
        """Adam with the step's coefficients read from the device buffer
        ``coef_dev`` (``gist_adam_update_dev``): what a replayed step uses."""
        for l in range(self.L):
            G.gist_adam_update_dev(self.ctx, params[l], self.dW[l], M[l], V[l], params[l].numel(),
                                   coef_dev, betas[0], betas[1], eps)

    def step(self, batch, params, lr, adam=None, loss_out=None):
        """``subTrain``: forward, loss, backward, update (all enqueued, nothing
        synced).  ``adam`` = (M, V, step, fresh) selects Adam, else SGD."""
        self.forward(batch, params)
        self.loss_and_grad(batch, loss_out)
        if adam is None:
            self.backward(batch, params, sgd_lr=lr)
        else:
            self.backward(batch, params)
            M, V, k, fresh = adam
            self.adam(params, M, V, lr, k, fresh)


class SubGCNBatch:
    """m sub-GCNs stepping on one shared mini-batch, as batched layer calls.

    The same arithmetic as m ``SubGCN`` steps on that batch, with one
    full-width aggregation per layer and grouped GEMMs (the layer
    descriptor's ``groups``).  The unpartitioned input is read once
    (``GIST_LAYER_SHARED_INPUT``: Abar X is formed once); hidden activations
    are n x (m s_l) with sub-GCN i in columns [i s_l, (i+1) s_l); the logits
    are group-major ([m][n][C]) so each sub-GCN's loss is one call.
    Parameters and gradients are per layer [m][rows][cols] tensors.
    """

    def __init__(self, ctx, kind, widths, m, n_cap, dtype=G.GIST_DTYPE_F32, device="cuda"):
        if kind not in ("gcn", "sage"):
            raise ValueError("batched sub-GCNs are GCN or SAGE")
        self.ctx = ctx
        self.kind = kind
        self.widths = list(widths)
        self.L = len(widths) - 1
        self.m = m
        self.dtype = dtype
        self.device = device
        self.lkind = G.GIST_LAYER_SAGE_MEAN if kind == "sage" else G.GIST_LAYER_GCN
        self.parts = 2 if kind == "sage" else 1
        self.n_cap = 0
        self.clustered = False   # the current batch is a cluster mini-batch
        self.ws = torch.empty(0, dtype=torch.uint8, device=device)
        self._alloc(n_cap)
        w = self.widths
        self.dW = [torch.empty(m, self.parts * w[l], w[l + 1], device=device) for l in range(self.L)]
        self.loss = torch.zeros(m, device=device)

    def _alloc(self, n_cap):
        w, d, m, L = self.widths, self.device, self.m, self.L
        self.n_cap = n_cap
        self.H = [None] + [torch.empty(n_cap, m * w[l + 1], device=d) for l in range(L - 1)]
        self.agg = [torch.empty(n_cap, w[0], device=d)] + \
                   [torch.empty(n_cap, m * w[l], device=d) for l in range(1, L)]
        self.dH = [None] + [torch.empty(n_cap, m * w[l], device=d) for l in range(1, L)]
        # group-major logits and their gradient: flat, viewed as [m][n][C] per batch
        self._logits = torch.empty(m * n_cap * w[L], device=d)
        self._dlogits = torch.empty(m * n_cap * w[L], device=d)
        self.loss_ws = torch.empty(G.gist_softmax_xent_workspace(n_cap), dtype=torch.uint8,
                                   device=d)

    def _gm(self, flat, n):
        C = self.widths[-1]
        return flat[:self.m * n * C].view(self.m, n, C)

    def _out(self, l, n):
        """Layer l's output for a batch of n rows (the last one group-major)."""
        return self.H[l + 1][:n] if l + 1 < self.L else self._gm(self._logits, n)

    def desc(self, l, n):
        act = G.GIST_ACT_RELU if l < self.L - 1 else G.GIST_ACT_NONE
        flags = (G.GIST_LAYER_SHARED_INPUT if l == 0 else 0) | \
                (G.GIST_LAYER_GROUP_MAJOR_OUT if l == self.L - 1 else 0) | \
                (G.GIST_LAYER_CLUSTERED if self.clustered else 0)
        return G.layer_desc(self.lkind, act, n, self.widths[l], self.widths[l + 1], self.dtype,
                            G.GIST_ORDER_AUTO, groups=self.m, flags=flags)

    def _workspace(self, n):
        need = 0
        for l in range(self.L):
            f, b = G.gist_layer_workspace_size(self.desc(l, n))
            need = max(need, f, b)
        if self.ws.numel() < need:
            self.ws = torch.empty(need, dtype=torch.uint8, device=self.device)
        return self.ws

    def logits(self, i):
        return self._gm(self._logits, self.n)[i]

    def forward(self, batch, params):
        n = batch.n
        if n > self.n_cap:
            raise ValueError("batch larger than the runner's capacity")
        self.n = n
        self.clustered = getattr(batch, "clustered", False)
        ws = self._workspace(n)
        H = batch.X
        for l in range(self.L):
            out = self._out(l, n)
            G.gist_gcn_layer_fwd(self.ctx, self.desc(l, n), batch.A, H, params[l],
                                 self.agg[l][:n], out, ws)
            H = out

    def loss_and_grad(self, batch):
        n, C = batch.n, self.widths[-1]
        logits, dlogits = self._gm(self._logits, n), self._gm(self._dlogits, n)
        for i in range(self.m):
            G.gist_softmax_xent(self.ctx, n, C, logits[i], batch.labels, self.loss[i:i + 1],
                                dlogits[i], self.loss_ws)

    def backward(self, batch, params, sgd_lr=None):
        """Every layer's backward pass into ``self.dW``, and with ``sgd_lr`` the
        SGD step fused into it (``gist_gcn_layer_bwd_sgd``, all m slices)."""
        fused = sgd_lr is not None
        n = batch.n
        ws = self._workspace(n)
        dout = self._gm(self._dlogits, n)
        for l in reversed(range(self.L)):
            Hin = batch.X if l == 0 else self.H[l][:n]
            dH = self.dH[l][:n] if l > 0 else None
            desc = self.desc(l, n)
            desc.flags |= relu_chain_flags(l, self.L)
            if fused:
                G.gist_gcn_layer_bwd_sgd(self.ctx, desc, batch.A, batch.A_T, Hin,
                                         self.agg[l][:n], self._out(l, n), params[l], dout,
                                         sgd_lr, dH, ws)
            else:
                G.gist_gcn_layer_bwd(self.ctx, desc, batch.A, batch.A_T, Hin,
                                     self.agg[l][:n], self._out(l, n), params[l], dout,
                                     self.dW[l], dH, ws)
            dout = dH
        if sgd_lr is not None and not fused:
            for l in range(self.L):
                G.gist_sgd_update(self.ctx, params[l], self.dW[l], params[l].numel(), sgd_lr)

    def step(self, batch, params, lr, adam=None):
        """All m sub-GCNs' ``subTrain`` step on the shared batch: SGD, or
        Adam with ``adam`` = (M, V, step, fresh) over the stacked moments."""
        self.forward(batch, params)
        self.loss_and_grad(batch)
        if adam is None:
            self.backward(batch, params, sgd_lr=lr)
            return
        self.backward(batch, params)
        M, V, k, fresh = adam
        for l in range(self.L):
            G.gist_adam_update(self.ctx, params[l], self.dW[l], M[l], V[l], params[l].numel(),
                               lr, k, flags=G.GIST_ADAM_FRESH if fresh else 0)


class GistModel:
    """Global parameters Theta on the device plus the subGCNs / subAgg calls.

    ``theta[l]`` is a list of parts, each with d_{l+1} columns: GCN
    [Theta_l]; SAGE [W_self, W_neigh]; GAT [Theta_l, A_l] with A_l the
    2 x d_{l+1} matrix whose rows are a_src and a_dst.  A sub-GCN's slice of
    a layer stacks its parts' slices row-wise in one (rows x s_{l+1}) matrix
    (the layout :class:`SubGCN` takes).  Rows of a weight part follow the
    partition D_l (all rows at l = 0); rows of GAT's attention part are
    never partitioned; columns follow D_{l+1} (all at the last layer).  A
    part split along neither (GAT's output-layer attention vectors) is
    trained in full by every sub-GCN and aggregated as the mean of the m
    copies (gist_subagg_mean); every other part is aggregated by
    replacement.

    A round is ``set_partitions`` -> ``begin_round`` -> m sub-GCN steps on
    ``params`` -> ``end_round``.  With ``fused`` (default) the subAgg of a
    round is deferred and performed by the next round's ``begin_round`` in
    the same pass over Theta as that round's gather (gist_subagg_gather);
    ``finalize`` applies a pending subAgg.  The slices are double-buffered
    so that the trained slices of round t and the gathered slices of round
    t+1 never share memory.

    ``adam`` adds Adam moments per slice (``M``, ``V``, same layout as
    ``params``).  The paper does not say what happens to them at subAgg:
    ``"carry"`` keeps global moments of Theta's shape that are gathered and
    aggregated exactly like the weights (in the same fused passes);
    ``"reset"`` restarts every sub-GCN's moments at each round (the caller
    passes ``fresh`` on its first local step), so no global moments exist.
    """

    def __init__(self, ctx, kind, widths, m, theta, device="cuda", fused=True, adam=None):
        if adam not in (None, "carry", "reset"):
            raise ValueError("adam is None, 'carry' or 'reset'")
        if kind not in ("gcn", "sage", "gat"):
            raise ValueError("kind is 'gcn', 'sage' or 'gat'")
        self.ctx = ctx
        self.kind = kind
        self.widths = list(widths)
        self.L = len(widths) - 1
        self.m = m
        self.theta = theta
        self.device = device
        self.fused = fused
        self.adam = adam
        self.parts = 1 if kind == "gcn" else 2
        self.slice_widths = [widths[0]] + [widths[l] // m for l in range(1, self.L)] + [widths[-1]]
        self.nbuf = 2 if fused else 1
        self._bufs = self._slices()                 # per sub-GCN parameter slices
        self._ptrs = self._tables(self._bufs)
        self._mbufs = self._vbufs = None
        self.Mg = self.Vg = None
        if adam:
            self._mbufs, self._vbufs = self._slices(), self._slices()
            self._mptrs, self._vptrs = self._tables(self._mbufs), self._tables(self._vbufs)
        if adam == "carry":
            self.Mg = [[torch.zeros_like(t) for t in parts] for parts in theta]
            self.Vg = [[torch.zeros_like(t) for t in parts] for parts in theta]
        self.buf = 0
        self._select(0)
        # two round slots of partition data: host (idx, offs); device
        # [idx; rank] (int32) and offs (int64)
        self._slot = 1
        self._host = [[None] * (self.L + 1) for _ in range(2)]
        self._pin = [[None] * (self.L + 1) for _ in range(2)]
        self._dev = [[None] * (self.L + 1) for _ in range(2)]
        self._doffs = [[None] * (self.L + 1) for _ in range(2)]
        self._events = [None, None]
        self._gevents = [None, None]   # gist events recorded after the partition uploads
        self.pending = None    # (slot, buffer) whose subAgg is outstanding

    # -- layout ---------------------------------------------------------------
    def _layout(self, l):
        """Layer l's parts: [(row offset in the slice, slice rows, global rows,
        rows follow D_l)]."""
        s = self.slice_widths[l]
        if self.kind == "gat":
            return [(0, s, self.widths[l], True), (s, 2, 2, False)]
        return [(p * s, s, self.widths[l], True) for p in range(self.parts)]

    def _row_split(self, l, p):
        return l > 0 and self._layout(l)[p][3]

    def _shared(self, l, p):
        """Split along neither dimension: every sub-GCN trains the whole part."""
        return not self._row_split(l, p) and l + 1 == self.L

    def _slice_rows(self, l):
        return sum(part[1] for part in self._layout(l))

    def _slices(self):
        """[buffer][sub-GCN][layer] slice tensors (parts stacked row-wise).

        Each (buffer, layer) is one [m][rows][cols] tensor and the per
        sub-GCN slices are views of it, so a batched step can address all m
        slices of a layer as one array (see ``stacked``)."""
        s = self.slice_widths
        big = [[torch.empty(self.m, self._slice_rows(l), s[l + 1], device=self.device)
                for l in range(self.L)] for _ in range(self.nbuf)]
        return [[[big[b][l][i] for l in range(self.L)] for i in range(self.m)]
                for b in range(self.nbuf)]

    def stacked(self, which="params"):
        """Per layer, the current buffer's [m][rows][cols] tensor of all slices."""
        bufs = {"params": self.params, "M": self.M, "V": self.V}[which]
        out = []
        for l in range(self.L):
            t = bufs[0][l]
            out.append(torch.as_strided(t, (self.m,) + tuple(t.shape),
                                        (t.numel(),) + tuple(t.stride())))
        return out

    def _tables(self, bufs):
        """Device tables of the m slice pointers of every (buffer, layer, part)."""
        s = self.slice_widths
        return [[[torch.tensor([bufs[b][i][l].data_ptr() + 4 * off * s[l + 1]
                                for i in range(self.m)], dtype=torch.int64).to(self.device)
                  for off, _, _, _ in self._layout(l)] for l in range(self.L)]
                for b in range(self.nbuf)]

    def _select(self, b):
        self.buf = b
        self.params = self._bufs[b]
        self.M = self._mbufs[b] if self._mbufs else None
        self.V = self._vbufs[b] if self._vbufs else None

    def _globals(self):
        """(global matrices, slice pointer tables, slice buffers) that gather /
        subAgg move."""
        out = [(self.theta, self._ptrs, self._bufs)]
        if self.adam == "carry":
            out += [(self.Mg, self._mptrs, self._mbufs), (self.Vg, self._vptrs, self._vbufs)]
        return out

    def _pairs(self, i):
        """(global matrices, sub-GCN i's slices of the current buffer) pairs."""
        out = [(self.theta, self.params[i])]
        if self.adam == "carry":
            out += [(self.Mg, self.M[i]), (self.Vg, self.V[i])]
        return out

    # -- partitions ---------------------------------------------------------
    def set_partitions(self, seeds):
        """``subGCNs`` partitions of every hidden width; ``seeds[l]`` for l = 1..L-1.

        Indices, ranks and offsets go through pinned buffers with
        asynchronous uploads, so the host does not wait for earlier rounds.
        """
        slot = 1 - self._slot
        if self._events[slot] is not None:
            self._events[slot].synchronize()   # the pinned buffers' last upload is done
        m = self.m
        if self._gevents[slot] is None:
            self._gevents[slot] = G.Event()
        for l in range(1, self.L):
            d = self.widths[l]
            if self._pin[slot][l] is None:
                # int32 [idx; rank] followed by the int64 offsets (as 2(m+1) int32), the
                # same layout on both sides so that one copy moves all three
                n32 = 2 * d + 2 * (m + 1)
                self._pin[slot][l] = torch.empty(n32, dtype=torch.int32, pin_memory=True)
                buf = torch.empty(n32, dtype=torch.int32, device=self.device)
                self._dev[slot][l] = buf[:2 * d].view(2, d)
                self._doffs[slot][l] = buf[2 * d:].view(torch.int64)
            idx, offs = G.gist_partition(d, m, seeds[l])
            rank = G.gist_partition_inverse(idx, offs)
            h = self._pin[slot][l].numpy()
            h[:d], h[d:2 * d] = idx, rank
            h[2 * d:].view(np.int64)[:] = offs
            self._host[slot][l] = (idx, offs)
            # the event after the last layer's copy marks the pinned buffers free
            G.gist_copy(self.ctx, self._dev[slot][l], self._pin[slot][l], 8 * d + 8 * (m + 1),
                        self._gevents[slot] if l == self.L - 1 else None)
        if self.L == 1:
            G.gist_copy(self.ctx, None, None, 0, self._gevents[slot])
        self._events[slot] = self._gevents[slot]
        self._slot = slot

    def _block(self, l, i):
        idx, offs = self._host[self._slot][l]
        return self._dev[self._slot][l][0][int(offs[i]):int(offs[i + 1])], int(offs[i + 1] - offs[i])

    def _rc(self, l, i, p):
        """(rows, nr, cols, nc) of sub-GCN i's slice of layer l, part p."""
        nrows = self._layout(l)[p][1]
        rows, nr = self._block(l, i) if self._row_split(l, p) else (None, nrows)
        if l + 1 == self.L:
            cols, nc = None, self.widths[-1]
        else:
            cols, nc = self._block(l + 1, i)
        return rows, nr, cols, nc

    def _set(self, slot, table, l, p):
        """gist_slice_set of layer l, part p: partition `slot`, slice pointer `table`."""
        rr = ro = cr = co = None
        if self._row_split(l, p):
            rr, ro = self._dev[slot][l][1], self._doffs[slot][l]
        if l + 1 < self.L:
            cr, co = self._dev[slot][l + 1][1], self._doffs[slot][l + 1]
        return G.slice_set(rr, ro, cr, co, table[l][p], self.slice_widths[l + 1])

    def _view(self, sl, l, p):
        off, nrows = self._layout(l)[p][:2]
        return sl[l][off:off + nrows]

    # -- per-slice calls ----------------------------------------------------
    def gather(self, i):
        """Theta^(i)_l = Theta_l[D_l^(i), D_{l+1}^(i)] for every layer and part
        (and the moments' slices with "carry")."""
        for glob, sl in self._pairs(i):
            for l in range(self.L):
                for p in range(self.parts):
                    rows, nr, cols, nc = self._rc(l, i, p)
                    G.gist_gather_slice(self.ctx, glob[l][p], self.widths[l + 1], rows, nr,
                                        cols, nc, self._view(sl, l, p), nc)

    def subagg(self, i, flags=0):
        """Write sub-GCN i's trained slices back into Theta (replacement);
        parts split along neither dimension wait for :meth:`subagg_shared`."""
        for glob, sl in self._pairs(i):
            for l in range(self.L):
                for p in range(self.parts):
                    if self._shared(l, p):
                        continue
                    rows, nr, cols, nc = self._rc(l, i, p)
                    G.gist_subagg(self.ctx, glob[l][p], self.widths[l + 1], rows, nr, cols,
                                  nc, self._view(sl, l, p), nc, flags)

    def subagg_shared(self, buf=None):
        """Unsplit parts: Theta's entries become the mean of the m trained copies
        of slice buffer ``buf`` (default: the current one)."""
        buf = self.buf if buf is None else buf
        for glob, tables, _ in self._globals():
            for l in range(self.L):
                for p in range(self.parts):
                    if self._shared(l, p):
                        grows = self._layout(l)[p][2]
                        G.gist_subagg_mean(self.ctx, glob[l][p], grows, self.widths[l + 1],
                                           self.widths[l + 1], self.m, tables[buf][l][p],
                                           self.slice_widths[l + 1])

    def _gather_shared(self, buf):
        """Every sub-GCN's copy of each unsplit part, into slice buffer ``buf``."""
        for glob, _, bufs in self._globals():
            for l in range(self.L):
                for p in range(self.parts):
                    if self._shared(l, p):
                        grows = self._layout(l)[p][2]
                        for i in range(self.m):
                            G.gist_gather_slice(self.ctx, glob[l][p], self.widths[l + 1], None,
                                                grows, None, self.widths[l + 1],
                                                self._view(bufs[buf][i], l, p),
                                                self.slice_widths[l + 1])

    # -- rounds ---------------------------------------------------------------
    def begin_round(self):
        """Gather this round's slices (after any pending subAgg of the last one)."""
        if not self.fused:
            for i in range(self.m):
                self.gather(i)
            return
        self._begin_state(self._begin_launches())

    def _begin_launches(self):
        """The launches of a fused :meth:`begin_round` (pending subAgg with this
        round's gather), in order; returns the slice buffer they fill."""
        nxt = 1 - self.buf if self.pending is not None else self.buf
        if self.pending is not None:
            self.subagg_shared(self.pending[1])
        for glob, tables, _ in self._globals():
            for l in range(self.L):
                for p in range(self.parts):
                    if self._shared(l, p):
                        continue
                    done = (self._set(self.pending[0], tables[self.pending[1]], l, p)
                            if self.pending is not None else None)
                    G.gist_subagg_gather(self.ctx, glob[l][p], self._layout(l)[p][2],
                                         self.widths[l + 1], self.widths[l + 1], self.m, done,
                                         self._set(self._slot, tables[nxt], l, p))
        self._gather_shared(nxt)
        return nxt

    def _begin_state(self, nxt):
        """The bookkeeping of a fused :meth:`begin_round`: slice buffer ``nxt``
        becomes the sub-GCNs' parameters, nothing is pending."""
        self._select(nxt)
        self.pending = None

    def end_round(self):
        """subAgg of this round's trained slices (deferred when fused)."""
        if not self.fused:
            for i in range(self.m):
                self.subagg(i)
            self.subagg_shared()
            return
        self.pending = (self._slot, self.buf)

    def finalize(self):
        """Apply a pending subAgg so that Theta holds every trained slice."""
        if self.pending is None:
            return
        self.subagg_shared(self.pending[1])
        for glob, tables, _ in self._globals():
            for l in range(self.L):
                for p in range(self.parts):
                    if self._shared(l, p):
                        continue
                    G.gist_subagg_gather(self.ctx, glob[l][p], self._layout(l)[p][2],
                                         self.widths[l + 1], self.widths[l + 1], self.m,
                                         self._set(self.pending[0], tables[self.pending[1]], l, p),
                                         None)
        self.pending = None


def gist_train(model, runner, rounds, zeta, lr, partition_seeds, batch, after_step=None):
    """Algorithm 1 on one device: ``rounds`` synchronisation rounds, each
    ``subGCNs`` -> ``zeta`` local steps per sub-GCN (``subTrain``, back to
    back) -> ``subAgg``.

    ``partition_seeds(t)`` -> {l: seed} for the hidden widths;
    ``batch(t, i, z)`` -> the loaded mini-batch of sub-GCN i's step z.
    The optimizer is the model's: SGD, or Adam with the bias correction
    counting every local step so far ("carry": k = t zeta + z + 1) or the
    round's steps ("reset": k = z + 1, moments restarted at z = 0).
    ``after_step(t, i, z, b)``, if given, is called after each local step is
    launched (for instance to read the runner's activations of batch ``b``).
    Returns the device tensor of losses [rounds, m, zeta]; nothing is synced.
    """
    losses = torch.empty(rounds, model.m, zeta, device=model.device)
    for t in range(rounds):
        model.set_partitions(partition_seeds(t))
        model.begin_round()
        for i in range(model.m):
            for z in range(zeta):
                b = batch(t, i, z)
                opt = None
                if model.adam == "carry":
                    opt = (model.M[i], model.V[i], t * zeta + z + 1, False)
                elif model.adam == "reset":
                    opt = (model.M[i], model.V[i], z + 1, z == 0)
                runner.step(b, model.params[i], lr, adam=opt, loss_out=losses[t, i, z:z + 1])
                if after_step is not None:
                    after_step(t, i, z, b)
        model.end_round()
    model.finalize()
    return losses
