"""The mini-batch pipeline (host CSR builds on worker threads into a ring of
pinned staging slots, uploads when taken) yields exactly the batches that
sequential ``BatchSlot.load`` calls produce: the CSR (and the SAGE
transpose) bit for bit, labels and gathered feature rows -- also when the
sequence is longer than the ring, so every slot is reused while its last
batch may still be in flight, and when a consumer enqueues work on a batch
before taking the next."""

import numpy as np
import pytest

from gist_synth.graphs import sbm

from gpu_util import log, to_dev, to_host

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("norm,depth,workers", [("gcn", 3, 2), ("sage", 2, 4), ("gcn", 8, 4)])
def test_pipeline_matches_sequential_loads(norm, depth, workers):
    import torch
    from paper_2102_10424_amd import gist as G
    from paper_2102_10424_amd.step import BatchPipeline, BatchSlot
    ctx = G.Context(0)
    g = sbm(3000, 30, 12.0, 0.9, 4)
    gh = G.GraphHandle(g)
    rng = np.random.default_rng(1)
    X = rng.standard_normal((g.n, 20)).astype(np.float32)
    y = rng.integers(0, 5, g.n).astype(np.int32)
    Xd = to_dev(X)
    order = [np.sort(rng.choice(30, int(rng.integers(1, 6)), replace=False)).astype(np.int32)
             for _ in range(11)]
    cap_n = int(np.sort(np.diff(g.cluster_ptr))[-5:].sum())
    cap_nnz = int(np.sort(np.diff(g.rowptr))[-cap_n:].sum()) + cap_n
    keys = ["rowptr", "col", "val"] + (["t_rowptr", "t_col", "t_val"] if norm == "sage" else [])
    ref = BatchSlot(ctx, norm, cap_n, cap_nnz, 20)
    want = []
    for cl in order:
        b = ref.load(gh, cl, Xd, y)
        torch.cuda.synchronize()
        n, nnz = b.n, b.nnz
        want.append(dict(n=n, nnz=nnz, X=to_host(b.X), labels=to_host(b.labels),
                         **{k: to_host(ref.d[k][:(n + 1 if k.endswith("rowptr") else nnz)])
                            for k in keys}))
    log(f"pipeline {norm} depth={depth} workers={workers}: {len(order)} batches")
    pipe = BatchPipeline(ctx, norm, cap_n, cap_nnz, 20, gh, Xd, y, order, depth=depth,
                         workers=workers)
    scratch = torch.empty(cap_n, 20, device="cuda")
    got = []
    for j in range(len(order)):
        b = pipe.next()
        scratch[:b.n].copy_(b.X)          # work on the batch, enqueued before the next is taken
        scratch[:b.n].mul_(2.0)
        slot = pipe.slots[j % depth]
        got.append(dict(n=b.n, nnz=b.nnz, X=to_host(scratch[:b.n]) / 2.0,
                        labels=to_host(b.labels),
                        **{k: to_host(slot.d[k][:(b.n + 1 if k.endswith("rowptr") else b.nnz)])
                           for k in keys}))
    pipe.close()
    for j, (a, w) in enumerate(zip(got, want)):
        assert (a["n"], a["nnz"]) == (w["n"], w["nnz"]), j
        for k in keys + ["labels", "X"]:
            assert np.array_equal(np.asarray(a[k]).view(np.uint32) if a[k].dtype == np.float32
                                  else a[k], np.asarray(w[k]).view(np.uint32)
                                  if w[k].dtype == np.float32 else w[k]), (j, k)
