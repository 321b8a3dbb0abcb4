#!/usr/bin/env python3
"""Benchmark: one GIST round of the ultra-wide GraphSAGE-mean workload on one GPU.

Workload (default ``--config c4``): 4-layer GraphSAGE-mean, hidden width
32,768 split into m = 8 sub-GCNs of 4,096, on a 2,449,029-node stochastic
block model (15,000 blocks, ~61.9M edges, 100 input features, 47 classes).
One timed step is one pass of the whole hot path:

  subGCNs partition of the three hidden widths (host)
  -> one pass over the 16 GiB global model that applies the previous
     round's subAgg and gathers all 8 sub-GCN weight slices (device)
  -> for each sub-GCN: cluster mini-batch of 10 blocks (host CSR build into
     pinned memory on worker threads, a few batches ahead of use;
     asynchronous upload, device feature-row gather),
     forward through 4 layers, softmax cross-entropy, backward, SGD.
  The last round's subAgg is applied after the timed region.

Inputs are seeded synthetic data resident in HBM before timing starts.
The reported value is ms per sub-GCN step = round time / (m zeta), with zeta
local steps per sub-GCN per round (default 1; ``--optimizer adam`` trains
with Adam as the paper's experiments do, its moments carried with the
weights through subAgg or reset each round).  The timed rounds carry no
per-kernel instrumentation: a HIP event at every round boundary gives the
per-round times (p10 / p50 / p90).  Kernel times come from a separate pass
of the same number of rounds in which the library records HIP event pairs
on the launch stream around every launch (gist_profile_*).  The default c4
run then measures, outside the timed region, the two other figures the
targets name: the full-graph aggregation of c5 (against HBM bandwidth) and
the bf16-input hidden-layer GEMMs of c4 (against the bf16 MFMA peak).  The
CPU baseline is the fp64 oracle timed on one sub-GCN step of the same
workload (and, with the extra figures, on the whole c5 aggregation).

Prints ONE JSON line.  ``--gpus N`` with N > 1 exits: the benchmark runs on
exactly one GPU.
"""

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK = {"f32": 157.3, "bf16": 2516.6}   # dense MFMA TFLOP/s, MI355X
CSRC = os.path.join(ROOT, "paper_2102_10424_amd", "csrc")
PROFILES = os.path.join(ROOT, "profiles")


def kernel_source_hash():
    """sha256 over the library's kernel and host sources (names and bytes)."""
    import hashlib
    h = hashlib.sha256()
    for f in sorted(os.listdir(CSRC)):
        if f.endswith((".hip", ".h", ".cuh", ".cpp")):
            h.update(f.encode())
            h.update(open(os.path.join(CSRC, f), "rb").read())
    return h.hexdigest()


def recorded_traffic(variant, workload, dtype):
    """Calibrated HBM bytes per launch of `variant` from the rocprofv3 counter
    records under profiles/ -- only if they were taken on these very sources."""
    if not os.path.isdir(PROFILES):
        return None
    src = kernel_source_hash()
    for f in sorted(os.listdir(PROFILES)):
        if not f.endswith(".md"):
            continue
        block = False
        for line in open(os.path.join(PROFILES, f)):
            if line.startswith("```traffic"):
                block = True
            elif line.startswith("```"):
                block = False
            elif block:
                r = json.loads(line)
                if (r["variant"], r["workload"], r["dtype"], r["src_sha256"]) == (
                        variant, workload, dtype, src):
                    return r["fetch_bytes"] + r["write_bytes"]
    return None
HBM_PEAK_GBS = 8000.0
METRIC = "sub-GCN fwd+bwd step ms; SpMM GB/s and GEMM TFLOP/s as % of MI355X peak"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default="c4",
                    choices=["c1", "c2", "c3", "c4", "c5", "c6", "c7"])
    ap.add_argument("--dtype", default="f32", choices=["f32", "bf16"])
    ap.add_argument("--d-in", type=int, default=256, help="c5 input slice width")
    ap.add_argument("--lr", type=float, default=0.01)
    ap.add_argument("--optimizer", default="sgd", choices=["sgd", "adam"],
                    help="sub-GCN update (c1-c4): SGD, or Adam as in the paper's experiments")
    ap.add_argument("--adam-policy", default="carry", choices=["carry", "reset"],
                    help="Adam moments at subAgg: carried with the weights, or reset per round")
    ap.add_argument("--zeta", type=int, default=1, help="local steps per sub-GCN per round")
    ap.add_argument("--streams", type=int, default=1,
                    help="HIP streams the m sub-GCN steps of a round are spread over")
    ap.add_argument("--shared-batch", action="store_true",
                    help="all m sub-GCNs step on one shared mini-batch, as batched layer calls")
    ap.add_argument("--graphs", action="store_true",
                    help="replay every sub-GCN step from a HIP graph (SGD, a mini-batch per "
                         "sub-GCN: cluster or LADIES batches at fixed padded shapes)")
    ap.add_argument("--round-graphs", action="store_true",
                    help="with --graphs: replay each whole round (fused subAgg + gather and "
                         "the m sub-GCN steps) from one HIP graph (SGD, zeta 1, one stream; "
                         "at least 5 warm-up rounds, which record the graphs)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true",
                    help="skip the library's per-launch event timing")
    ap.add_argument("--copy-calib", action="store_true",
                    help="only run a plain 1 GiB row copy (counter calibration)")
    ap.add_argument("--loss-curves", action="store_true",
                    help="only train GIST with Adam for m in {1, 2, 4, 8} and both moment "
                         "policies on a learnable c3-graph task and print the loss per round")
    ap.add_argument("--curve-rounds", type=int, default=20)
    ap.add_argument("--curve-zeta", type=int, default=10)
    ap.add_argument("--aggregation", default="tile", choices=["tile", "gather"],
                    help="cluster mini-batches and the c5 matrix: the matrix-core tiles of "
                         "GIST_LAYER_CLUSTERED (default), or the gather kernel")
    ap.add_argument("--curve-hidden", type=int, default=256)
    ap.add_argument("--curve-lr", type=float, default=0.01)
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the extra figures (c5 aggregation, c4 bf16 GEMMs) measured after "
                         "the timed region of the default c4 run")
    ap.add_argument("--profile-steps", type=int, default=0,
                    help="steps of the separate profiled pass (0: as many as --steps)")
    return ap.parse_args()


# ---------------------------------------------------------------------------
class RoundWorkload:
    """A GIST round (partition, gather, m sub-GCN steps, subAgg) on one GPU."""

    def __init__(self, cfg, ctx, dtype, optimizer="sgd", policy="carry", zeta=1, shared=False,
                 streams=1, graphs=False, lr=0.01, clustered=True, round_graphs=False):
        import torch
        from paper_2102_10424_amd import gist as G
        from paper_2102_10424_amd.step import (BatchPipeline, BatchSlot, ClusterGraphRunner,
                                               FixedBatchSlot, GistModel, LadiesGraphRunner,
                                               RoundReplayer, SubGCN, SubGCNBatch)
        self.cfg, self.ctx, self.G = cfg, ctx, G
        self.lr = lr
        self.adam = policy if optimizer == "adam" else None
        self.use_graphs = self.graphs = graphs
        t0 = time.time()
        self.graph = cfg.make_graph()
        log(f"[bench] graph n={self.graph.n} nnz={self.graph.nnz} ({time.time() - t0:.1f}s)")
        self.gh = G.GraphHandle(self.graph)
        self.X = torch.from_numpy(cfg.features_matrix()).cuda()
        self.labels = cfg.labels()
        theta = []
        t0 = time.time()
        for l in range(cfg.L):
            parts = []
            for p in range(cfg.n_parts()):
                parts.append(torch.from_numpy(cfg.theta(l, p)).cuda())
            theta.append(parts)
        log(f"[bench] global theta on device ({time.time() - t0:.1f}s)")
        self.zeta = zeta
        self.model = GistModel(ctx, cfg.kind, cfg.widths, cfg.m, theta, adam=self.adam)
        self.norm = "sage" if cfg.kind == "sage" else "gcn"
        self.ladies = cfg.ladies
        if self.ladies and shared:
            raise ValueError("LADIES mini-batches are per sub-GCN (no shared batch)")
        if graphs and (shared or not (self.ladies or cfg.batch_clusters)):
            raise ValueError("--graphs replays sub-GCN steps on per-sub-GCN mini-batches")
        if round_graphs and not (graphs and streams == 1 and zeta == 1 and self.adam is None):
            raise ValueError("--round-graphs needs --graphs, SGD, zeta 1 and one stream")
        self.round_graphs = round_graphs
        # round replays read each round's m mini-batches from the same pipeline
        # slots every fourth round: a ring of 4m slots (three rounds of builds
        # ahead; with 2m the builds fell behind)
        ring = 4 * cfg.m if round_graphs else 12
        # capacities: the largest mini-batch of the clusters, generous nnz bound
        if self.ladies:
            cap_n = self.ladies["batch"] + cfg.L * self.ladies["samples"]
            cap_nnz = 0
        elif cfg.batch_clusters is None:
            cap_n = self.graph.n
            cap_nnz = self.graph.nnz + self.graph.n
        else:
            sizes = np.diff(self.graph.cluster_ptr)
            cap_n = int(np.sort(sizes)[-cfg.batch_clusters:].sum())
            cap_nnz = int(np.sort(np.diff(self.graph.rowptr))[-cap_n:].sum()) + cap_n
        self.full = None
        self.pipe = None
        # sub-GCN i of a round runs on stream i mod streams (its own context,
        # runner buffers and mini-batch pipeline); stream 0 is torch's current
        self.nstreams = 1 if shared else max(1, streams)
        self.streams = [torch.cuda.current_stream()] + [torch.cuda.Stream()
                                                         for _ in range(self.nstreams - 1)]
        self.ctxs = [ctx] + [G.Context(0, stream=st.cuda_stream) for st in self.streams[1:]]
        if self.ladies:
            # LADIES mini-batches sampled from the full-graph GCN matrix on host workers
            t0 = time.time()
            self.A_full = G.CsrHandle(G.gist_build_minibatch_csr(self.graph, None, "gcn"))
            max_deg = int(np.max(np.diff(self.graph.rowptr)))
            log(f"[bench] full GCN matrix nnz={self.A_full.nnz} ({time.time() - t0:.1f}s)")
            self.pipes = [BatchPipeline.ladies(c, cfg.L, self.ladies["batch"],
                                               self.ladies["samples"], max_deg, cfg.widths[0],
                                               self.A_full, self.X, self.labels,
                                               self._ladies_order(zeta, k, self.nstreams),
                                               depth=ring if graphs else 8,
                                               workers=(12 if graphs else 8) // self.nstreams,
                                               fixed=graphs)
                          for k, c in enumerate(self.ctxs)]
            self.pipe = self.pipes[0]
        elif cfg.batch_clusters is None:
            self.slots = [BatchSlot(ctx, self.norm, cap_n, cap_nnz, cfg.widths[0])]
        else:
            # mini-batches are built on host worker threads ahead of use
            self.pipes = [BatchPipeline(c, self.norm, cap_n, cap_nnz, cfg.widths[0], self.gh,
                                        self.X, self.labels,
                                        self._cluster_order(shared, zeta, k, self.nstreams),
                                        depth=8, workers=(12 if graphs else 4) // self.nstreams,
                                        slots=[FixedBatchSlot(c, self.norm, cap_n, cap_nnz,
                                                              cfg.widths[0], clustered=clustered)
                                               for _ in range(ring if graphs else 8)],
                                        build=self._fixed_build)
                          for k, c in enumerate(self.ctxs)]
            self.pipe = self.pipes[0]
        dt = G.GIST_DTYPE_BF16_IN if dtype == "bf16" else G.GIST_DTYPE_F32
        self.shared = shared
        if shared:
            self.runner = SubGCNBatch(ctx, cfg.kind, self.model.slice_widths, cfg.m, cap_n, dtype=dt)
        else:
            self.runners = [SubGCN(c, cfg.kind, self.model.slice_widths, cap_n, dtype=dt)
                            for c in self.ctxs]
            self.runner = self.runners[0]
            if graphs and self.ladies:
                self.graph_runners = [
                    LadiesGraphRunner(c, self.model.slice_widths, cfg.L, self.ladies["batch"],
                                      self.ladies["samples"], cfg.widths[0], self.X, dtype=dt)
                    for c in self.ctxs]
            elif graphs:
                self.graph_runners = [
                    ClusterGraphRunner(c, cfg.kind, self.model.slice_widths, cap_n, cap_nnz,
                                       cfg.widths[0], self.X, dtype=dt, clustered=clustered)
                    for c in self.ctxs]
            if round_graphs:
                self.round_replayer = RoundReplayer(self.model, self.graph_runners[0],
                                                    self.pipes[0], lr)
        self.t = 0

    def _coef(self, t, z):
        """Adam coefficients of local step z of round t (a replayed Adam step
        reads them from its batch), or None."""
        if not (self.graphs and self.adam):
            return None
        carry = self.adam == "carry"
        k = t * self.zeta + z + 1 if carry else z + 1
        flags = self.G.GIST_ADAM_FRESH if (not carry and z == 0) else 0
        return self.G.gist_adam_coefficients(self.lr, k, flags=flags)

    def _cluster_order(self, shared, zeta, k=0, nstreams=1):
        """The clusters of every mini-batch of stream k, in the order the
        rounds take them (sub-GCNs k, k + nstreams, ...), with the step's Adam
        coefficients."""
        cfg, t = self.cfg, 0
        while True:
            for i in range(k, 1 if shared else cfg.m, nstreams):
                for z in range(zeta):
                    yield (lambda t=t, i=i, z=z: (cfg.minibatch(t, i, z), self._coef(t, z)))
            t += 1

    def _fixed_build(self, slot, item):
        clusters, coef = item()
        slot.build(self.gh, clusters, self.labels, coef=coef)

    def _ladies_order(self, zeta, k=0, nstreams=1):
        """Every LADIES mini-batch of stream k, as a callable the pipeline's
        worker evaluates to (output nodes, draw seed)."""
        cfg, t = self.cfg, 0
        while True:
            for i in range(k, cfg.m, nstreams):
                for z in range(zeta):
                    yield (lambda t=t, i=i, z=z: (cfg.ladies_batch(t, i, z),
                                                  cfg.ladies_seed(t, i, z), self._coef(t, z)))
            t += 1

    def _batch(self, t, i, z, k=0):
        if self.cfg.batch_clusters is None and not self.ladies:
            if self.full is None:
                self.full = self.slots[0].load(self.gh, None, self.X, self.labels)
            return self.full
        return self.pipes[k].next()

    def step(self):
        cfg, m = self.cfg, self.model
        t, zeta = self.t, self.zeta
        if self.use_graphs and self.round_graphs:
            self.round_replayer.round({l: cfg.partition_seed(t, l) for l in range(1, cfg.L)})
            self.t += 1
            return
        m.set_partitions({l: cfg.partition_seed(t, l) for l in range(1, cfg.L)})
        m.begin_round()   # subAgg of round t-1 fused with the gather of round t
        if self.shared:
            for z in range(zeta):
                b = self._batch(t, 0, z)
                opt = None
                if self.adam:
                    k = t * zeta + z + 1 if self.adam == "carry" else z + 1
                    opt = (m.stacked("M"), m.stacked("V"), k, self.adam == "reset" and z == 0)
                self.runner.step(b, m.stacked(), self.lr, adam=opt)
            m.end_round()
            self.t += 1
            return
        import torch
        if self.nstreams > 1:   # the other streams start after the fused pass
            ev = torch.cuda.Event()
            ev.record(self.streams[0])
            for st in self.streams[1:]:
                st.wait_event(ev)
        for i in range(cfg.m):
            k = i % self.nstreams
            with torch.cuda.stream(self.streams[k]):
                if self.use_graphs:
                    gr = self.graph_runners[k]
                    adam = (m.M[i], m.V[i]) if self.adam else None
                    for z in range(zeta):
                        self.pipes[k].take(lambda slot: gr.step(slot, m.params[i], self.lr, adam))
                    continue
                for z in range(zeta):
                    b = self._batch(t, i, z, k)
                    opt = None
                    if self.adam == "carry":
                        opt = (m.M[i], m.V[i], t * zeta + z + 1, False)
                    elif self.adam == "reset":
                        opt = (m.M[i], m.V[i], z + 1, z == 0)
                    self.runners[k].step(b, m.params[i], self.lr, adam=opt)
        for st in self.streams[1:]:   # subAgg waits for every stream's steps
            ev = torch.cuda.Event()
            ev.record(st)
            self.streams[0].wait_event(ev)
        m.end_round()
        self.t += 1

    def finish(self):
        self.model.finalize()
        for p in getattr(self, "pipes", []):
            p.close()

    def steps_per_unit(self):
        return self.cfg.m * self.zeta

    def describe(self):
        c = self.cfg
        if self.ladies:
            batch = (f"LADIES mini-batch: {self.ladies['batch']} output nodes, "
                     f"{self.ladies['samples']} draws per layer")
        elif c.batch_clusters:
            batch = f"mini-batch {c.batch_clusters} clusters"
        else:
            batch = "full graph"
        return {"workload": f"{c.name}: GIST round, {c.L}-layer "
                            f"{dict(sage='GraphSAGE-mean', gcn='GCN', gat='GAT')[c.kind]}, hidden "
                            f"{c.widths[1]} split m={c.m}, N={c.n_nodes}, {batch}",
                "model": "GIST sub-GCN", "m": c.m, "widths": c.widths,
                "global_batch": (self.ladies["batch"] if self.ladies else
                                 c.batch_clusters or c.n_nodes), "zeta": self.zeta,
                "batching": "m sub-GCNs on one shared mini-batch (batched layers)" if self.shared
                            else "one mini-batch per sub-GCN",
                "optimizer": f"adam ({self.adam} moments)" if self.adam else "sgd",
                "launch": ("each round replayed from one HIP graph" if self.round_graphs else
                           "each sub-GCN step replayed from a HIP graph") if self.graphs
                          else "kernels launched one by one"}

    # ---- CPU baseline: the fp64 oracle on one sub-GCN step ---------------------
    def cpu_baseline(self):
        from oracle import gist as OG
        from oracle import minibatch as OM
        from oracle import partition as OP
        cfg = self.cfg
        parts = [None] * (cfg.L + 1)
        for l in range(1, cfg.L):
            parts[l] = OP.partition(cfg.widths[l], cfg.m, cfg.partition_seed(0, l))
        sl = OG.slice_indices(parts, cfg.L, 0)
        params = []
        for l, (r, c) in enumerate(sl):
            ps = []
            for p in range(cfg.n_parts()):
                rows = r if r is not None and not (cfg.kind == "gat" and p == 1) else None
                th = cfg.theta(l, p, rows=rows) if rows is not None else cfg.theta(l, p)
                ps.append(th if c is None else th[:, c])
            if cfg.kind == "gat":
                params.append((ps[0], ps[1][0], ps[1][1]))
            else:
                params.append(ps[0] if cfg.kind == "gcn" else (ps[0], ps[1]))
        if self.ladies:
            from oracle import ladies as OLD
            A = OM.build(self.graph, None, "gcn")
            t0 = time.time()
            smp = OLD.sample(A, cfg.ladies_batch(0, 0), cfg.L, self.ladies["samples"],
                             cfg.ladies_seed(0, 0))
            t_s = time.time() - t0
            csr = smp["layers"]
            X = cfg.features_matrix(rows=smp["nodes"][0])
            y = self.labels[smp["nodes"][cfg.L]]
        else:
            csr = OM.build(self.graph, cfg.minibatch(0, 0), self.norm)
            nm = csr["node_map"]
            X = cfg.features_matrix(rows=nm)
            y = self.labels[nm]
            t_s = 0.0
        t0 = time.time()
        OG.sub_gcn_step(cfg.kind, csr, X, y, params, self.lr)
        dt = time.time() - t0 + t_s
        return dt * 1e3, "one sub-GCN step (fwd + loss + bwd + SGD) of round 0, sub-GCN 0, " \
                         "fp64" + (", with its LADIES sampling" if self.ladies else "") + \
                         "; excludes partition, slice gather and subAgg"


class LayerWorkload:
    """c5: one GCN layer fwd+bwd over the whole graph (output slice of m=8)."""

    def finish(self):
        pass

    def __init__(self, cfg, ctx, dtype, d_in, clustered=True):
        import torch
        from paper_2102_10424_amd import gist as G
        from paper_2102_10424_amd.step import BatchSlot
        cfg.widths = [d_in, cfg.widths[1]]
        self.cfg, self.ctx, self.G = cfg, ctx, G
        self.d_in = d_in
        t0 = time.time()
        self.graph = cfg.make_graph()
        log(f"[bench] graph n={self.graph.n} nnz={self.graph.nnz} ({time.time() - t0:.1f}s)")
        gh = G.GraphHandle(self.graph)
        n = self.graph.n
        self.slot = BatchSlot(ctx, "gcn", n, self.graph.nnz + n, d_in, clustered=clustered)
        self.X = torch.from_numpy(cfg.features_matrix()).cuda()
        self.b = self.slot.load(gh, None, self.X, cfg.labels())
        torch.cuda.synchronize()
        idx, offs = G.gist_partition(cfg.widths[1], cfg.m, cfg.partition_seed(0, 1))
        cols = torch.from_numpy(idx[offs[0]:offs[1]].copy()).cuda()
        th = torch.from_numpy(cfg.theta(0, 0)).cuda()
        self.s_out = int(offs[1] - offs[0])
        self.W = torch.empty(d_in, self.s_out, device="cuda")
        G.gist_gather_slice(ctx, th, cfg.widths[1], None, d_in, cols, self.s_out, self.W,
                            self.s_out)
        self.dHo = torch.from_numpy(cfg.upstream(n, self.s_out)).cuda()
        self.desc = G.layer_desc(G.GIST_LAYER_GCN, G.GIST_ACT_RELU, n, d_in, self.s_out,
                                 G.GIST_DTYPE_BF16_IN if dtype == "bf16" else G.GIST_DTYPE_F32,
                                 flags=G.GIST_LAYER_CLUSTERED if clustered else 0)
        # backward as a hidden layer inside a ReLU chain: the upstream gradient
        # arrives as dZ (the layer above applied this layer's ReLU derivative)
        # and dH leaves times the layer below's derivative 1[H > 0]
        self.bdesc = G.layer_desc(G.GIST_LAYER_GCN, G.GIST_ACT_RELU, n, d_in, self.s_out,
                                  self.desc.dtype, flags=self.desc.flags | G.GIST_LAYER_DZ_IN |
                                  G.GIST_LAYER_MASK_DH)
        f, bb = G.gist_layer_workspace_size(self.desc)
        self.ws = torch.empty(max(f, bb), dtype=torch.uint8, device="cuda")
        self.agg = torch.empty(n, d_in, device="cuda")
        self.Ho = torch.empty(n, self.s_out, device="cuda")
        self.dW = torch.empty(d_in, self.s_out, device="cuda")
        self.dH = torch.empty(n, d_in, device="cuda")

    def step(self):
        G, b = self.G, self.b
        G.gist_gcn_layer_fwd(self.ctx, self.desc, b.A, b.X, self.W, self.agg, self.Ho, self.ws)
        G.gist_gcn_layer_bwd(self.ctx, self.bdesc, b.A, None, b.X, self.agg, self.Ho, self.W,
                             self.dHo, self.dW, self.dH, self.ws)

    def steps_per_unit(self):
        return 1

    def describe(self):
        return {"workload": f"c5: one GCN layer fwd+bwd, full graph N={self.graph.n}, "
                            f"nnz={self.graph.nnz + self.graph.n}, {self.d_in}->{self.s_out}; "
                            "backward as a hidden layer of a ReLU chain (dZ in, masked dH out)",
                "model": "GIST sub-GCN layer", "global_batch": self.graph.n,
                "d_in": self.d_in, "s_out": self.s_out}

    def cpu_baseline(self):
        """The oracle's forward of the whole layer, timed in full: fp64
        Abar H over all rows (the oracle's CSR, SciPy) and the transform with
        ReLU (NumPy BLAS).  The backward is not timed (it would double the
        run for the same kind of work); the sample field says so."""
        from oracle import layers as OL
        from oracle import minibatch as OM
        csr = OM.build(self.graph, None, "gcn")
        X = self.cfg.features_matrix()
        W = self.W.cpu().numpy()
        t0 = time.time()
        OL.gcn_forward(csr, X, W, True)
        dt = time.time() - t0
        return dt * 1e3, (f"fp64 forward of the whole layer ({csr['n']} rows, aggregation "
                          "with SciPy on one thread + transform and ReLU with NumPy BLAS), "
                          "timed in full; backward not timed")


def copy_calibration(G, ctx):
    """Plain copy of a known size: 16384 x 16384 fp32 (1 GiB read, 1 GiB written)
    through the library's row-copy kernel (gather with no index lists), three
    times.  HBM byte counters of these launches calibrate the counters read
    on the other kernels."""
    import torch
    n = 16384
    src = torch.randn(n, n, device="cuda")
    dst = torch.empty_like(src)
    G.gist_profile_begin(ctx, 16)
    for _ in range(3):
        G.gist_gather_slice(ctx, src, n, None, n, None, n, dst, n)
    prof, _ = G.gist_profile_read(ctx)
    G.gist_profile_end(ctx)
    v = prof["gather_slice"]
    print(json.dumps({"copy_bytes_read": n * n * 4, "copy_bytes_written": n * n * 4,
                      "launches": v["launches"], "avg_us": 1e3 * v["ms"] / v["launches"],
                      "gbs": v["bytes"] / (v["ms"] * 1e-3) / 1e9}), flush=True)


def cpu_info():
    """Host facts for the CPU baseline: logical CPUs, the CPU model and the
    threads the BLAS behind NumPy / SciPy actually uses."""
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    return {"cores": int(threads), "logical_cpus": os.cpu_count(), "cpu_model": model,
            "blas_threads": int(threads)}


def timed_pass(wl, steps):
    """K steps with no per-kernel instrumentation: a HIP event on the launch
    stream at every step boundary (per-step times), and the host clock around
    the whole pass between two device synchronisations (the mean)."""
    import torch
    st = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev[0].record(st)
    for s in range(steps):
        wl.step()
        ev[s + 1].record(st)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    return (t1 - t0) * 1e3 / steps, [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]


def merged_profile(G, ctxs):
    prof, dropped = {}, 0
    for c in ctxs:   # every stream's launches (their event times may overlap)
        p, d = G.gist_profile_read(c)
        G.gist_profile_end(c)
        dropped += d
        for k, v in p.items():
            acc = prof.setdefault(k, dict(launches=0, ms=0.0, flops=0.0, bytes=0.0))
            for f in acc:
                acc[f] += v[f]
    return prof, dropped


def is_gemm(name):
    return name.startswith("gemm_") and "reduce" not in name and "fixup" not in name


def hidden_gemms(prof, gflop, peak):
    """Per variant: rate of the launches that are the hidden layers' products
    (about `gflop` GFLOP each), as TFLOP/s and fraction of `peak`."""
    out = {}
    for k, v in prof.items():
        if not is_gemm(k) or not v["launches"]:
            continue
        per = v["flops"] / v["launches"] / 1e9
        if abs(per - gflop) > 0.02 * gflop:
            continue
        t = v["flops"] / (v["ms"] * 1e-3) / 1e12
        out[k] = {"tflops": round(t, 2), "frac": round(t / peak, 4), "launches": v["launches"],
                  "avg_launch_us": round(1e3 * v["ms"] / v["launches"], 2)}
    return out


def target_figures(wl, ctx, steps, clustered=True):
    """The two figures the default line does not time in its own workload,
    measured after the timed region: the full-graph aggregation of c5 (Abar H
    over the whole c4 graph, width 256, fp32) against HBM bandwidth, and the
    bf16-input hidden-layer GEMMs of c4 against the bf16 MFMA peak (sub-GCN
    steps on the round's own mini-batches and weights, on copies)."""
    import torch
    from paper_2102_10424_amd import gist as G
    from paper_2102_10424_amd.step import BatchSlot, SubGCN
    out = {}
    cfg = wl.cfg
    # --- c4 bf16 hidden GEMMs
    runner = SubGCN(ctx, cfg.kind, wl.model.slice_widths, wl.runner.n_cap,
                    dtype=G.GIST_DTYPE_BF16_IN)
    params = [p.clone() for p in wl.model.params[0]]
    b = wl.pipes[0].next()
    runner.step(b, params, wl.lr)       # warm-up: workspace and code objects
    torch.cuda.synchronize()
    G.gist_profile_begin(ctx, 1 << 14)
    for _ in range(steps):
        runner.step(wl.pipes[0].next(), params, wl.lr)
    torch.cuda.synchronize()
    prof, _ = merged_profile(G, [ctx])
    s = wl.model.slice_widths
    gf = 2.0 * 2 * s[1] * s[2] * 1633 / 1e9     # [H | Abar H] W at the mean batch size
    g = hidden_gemms(prof, 109.565, PEAK["bf16"]) or hidden_gemms(prof, gf, PEAK["bf16"])
    tot_f = sum(prof[k]["flops"] for k in g)
    tot_ms = sum(prof[k]["ms"] for k in g)
    out["gemm_c4_bf16"] = {
        "what": f"c4 hidden-layer products with bf16-input MFMA ({steps} sub-GCN steps on the "
                "round's mini-batches, copies of sub-GCN 0's slices; library HIP events)",
        "variants": g, "tflops": round(tot_f / (tot_ms * 1e-3) / 1e12, 2) if tot_ms else None,
        "peak": PEAK["bf16"], "unit": "TFLOP/s",
        "frac": round(tot_f / (tot_ms * 1e-3) / 1e12 / PEAK["bf16"], 4) if tot_ms else None,
        "target_frac": 0.5}
    del runner, params
    # --- c5 aggregation over the full graph, width 256
    n = wl.graph.n
    w = 256
    slot = BatchSlot(ctx, "gcn", n, wl.graph.nnz + n, w)
    gen = torch.Generator(device="cuda").manual_seed(105)
    X = torch.randn(n, w, device="cuda", generator=gen)
    bb = slot.load(wl.gh, None, X, wl.labels)
    desc = G.layer_desc(G.GIST_LAYER_GCN, G.GIST_ACT_RELU, n, w, w, G.GIST_DTYPE_F32,
                        G.GIST_ORDER_AGG_FIRST, flags=G.GIST_LAYER_CLUSTERED if clustered else 0)
    fws, bws = G.gist_layer_workspace_size(desc)
    ws = torch.empty(max(fws, bws, 1), dtype=torch.uint8, device="cuda")
    W = torch.randn(w, w, device="cuda", generator=gen) / 16.0
    agg = torch.empty(n, w, device="cuda")
    Ho = torch.empty(n, w, device="cuda")
    G.gist_gcn_layer_fwd(ctx, desc, bb.A, bb.X, W, agg, Ho, ws)
    torch.cuda.synchronize()
    G.gist_profile_begin(ctx, 1 << 10)
    for _ in range(steps):
        G.gist_gcn_layer_fwd(ctx, desc, bb.A, bb.X, W, agg, Ho, ws)
    torch.cuda.synchronize()
    prof, _ = merged_profile(G, [ctx])
    agg_k = {k: v for k, v in prof.items() if k.startswith("spmm")}
    a_ms = sum(v["ms"] for v in agg_k.values())
    a_bytes = sum(v["bytes"] for v in agg_k.values())
    launches = steps
    gbs = a_bytes / (a_ms * 1e-3) / 1e9 if a_ms else None
    out["spmm_c5"] = {
        "what": f"c5: Abar H over the full {n}-node GCN matrix ({bb.nnz} entries), width {w}, "
                f"fp32, {launches} calls (library HIP events; kernels: {sorted(agg_k)})",
        "achieved": round(gbs, 1) if gbs else None, "peak": HBM_PEAK_GBS, "unit": "GB/s",
        "frac": round(gbs / HBM_PEAK_GBS, 4) if gbs else None,
        "bytes_per_call": round(a_bytes / launches), "ms_per_call": round(a_ms / launches, 4),
        "target_frac": 0.6,
        "bytes_def": "4(n+1) + 8 nnz + 4 n w (X read once) + 4 n w (Y written once)"}
    del slot, X, bb, agg, Ho, ws
    torch.cuda.synchronize()
    out["library_gemm_c4"] = dict(
        what="torch.mm (vendor BLAS) on contiguous operands of the c4 hidden-layer shapes at the "
             "mean batch size, bf16 and fp32; context for gemm_c4_bf16 and the roofline GEMM, "
             "not part of the product path",
        **library_gemm_figures(1633, wl.model.slice_widths[1]))
    return out


def library_gemm_figures(m=1633, s=4096, reps=10):
    """Context for the GEMM figures: torch.mm (the vendor BLAS) on plain
    contiguous operands of the c4 hidden-layer shapes -- forward (m x 2s) @
    (2s x s), input gradient (m x s) @ (s x 2s), weight gradient (2s x m) @
    (m x s) -- in bf16 and in fp32 (TF32 off), timed with events on torch's
    stream.  No fused epilogue, no concatenated or transposed operands: a
    library reference point, not part of the product path."""
    import torch
    torch.backends.cuda.matmul.allow_tf32 = False
    shapes = {"forward": (m, s, 2 * s), "input_grad": (m, 2 * s, s), "weight_grad": (2 * s, s, m)}
    out = {}
    gen = torch.Generator(device="cuda").manual_seed(7)
    for dname, dt in (("bf16", torch.bfloat16), ("f32", torch.float32)):
        row = {}
        for name, (mm, nn, kk) in shapes.items():
            a = torch.randn(mm, kk, device="cuda", generator=gen).to(dt).contiguous()
            b = torch.randn(kk, nn, device="cuda", generator=gen).to(dt).contiguous()
            for _ in range(2):
                torch.mm(a, b)
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                torch.mm(a, b)
            e1.record()
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / reps
            tf = 2.0 * mm * nn * kk / (us * 1e-6) / 1e12
            row[name] = {"M": mm, "N": nn, "K": kk, "us": round(us, 1), "tflops": round(tf, 1),
                         "frac": round(tf / PEAK[dname], 4)}
            del a, b
        out[dname] = row
    return out


def c5_oracle_spmm_ms(graph, w=256):
    """The oracle's aggregation over the whole c5 matrix at width 256, timed
    in full (no extrapolation): fp64 Abar H with Abar from the oracle's own
    CSR build, as a SciPy CSR product on one thread."""
    import scipy.sparse as sp
    from oracle import minibatch as OM
    csr = OM.build(graph, None, "gcn")
    n = csr["n"]
    A = sp.csr_matrix((csr["val"].astype(np.float64), csr["col"], csr["rowptr"]), shape=(n, n))
    H = np.random.default_rng(105).standard_normal((n, w))
    t0 = time.perf_counter()
    A @ H
    return (time.perf_counter() - t0) * 1e3


def oracle_single_thread_ms(names=("c1", "c2", "c3")):
    """The oracle's sub-GCN step (fwd + loss + bwd + SGD; round 0, sub-GCN 0,
    fp64) on the small workloads with the BLAS behind NumPy / SciPy held to
    one thread (threadpoolctl); graph, batch and parameters are built
    outside the timed region."""
    from threadpoolctl import threadpool_limits
    from gist_synth import get_config
    from oracle import gist as OG
    from oracle import minibatch as OM
    from oracle import partition as OP
    out = {}
    for name in names:
        cfg = get_config(name)
        graph = cfg.make_graph()
        parts = [None] * (cfg.L + 1)
        for l in range(1, cfg.L):
            parts[l] = OP.partition(cfg.widths[l], cfg.m, cfg.partition_seed(0, l))
        params = []
        for l, (r, c) in enumerate(OG.slice_indices(parts, cfg.L, 0)):
            ps = []
            for p in range(cfg.n_parts()):
                th = cfg.theta(l, p, rows=r) if r is not None else cfg.theta(l, p)
                ps.append(th if c is None else th[:, c])
            params.append(ps[0] if cfg.kind == "gcn" else (ps[0], ps[1]))
        mb = cfg.minibatch(0, 0) if cfg.batch_clusters is not None else None
        csr = OM.build(graph, mb, "sage" if cfg.kind == "sage" else "gcn")
        nm = csr.get("node_map")
        X = cfg.features_matrix(rows=nm) if nm is not None else cfg.features_matrix()
        y = cfg.labels()
        y = y[nm] if nm is not None else y
        with threadpool_limits(limits=1):
            t0 = time.perf_counter()
            OG.sub_gcn_step(cfg.kind, csr, X, y, params, 0.01)
            out[name] = round((time.perf_counter() - t0) * 1e3, 1)
    return out


def loss_curves(G, ctx, rounds, zeta, lr=0.01, hidden=256, eval_clusters=40):
    """Algorithm 1 trained with Adam (the paper's optimizer, no weight decay)
    for m = 1 (the full model), 2, 4 and 8, with the moments carried through
    subAgg or reset each round, on the c3 graph (232,965 nodes, 1,500
    clusters, 20 per mini-batch) and a 3-layer GraphSAGE-mean 602-h-h-41.

    Uniformly random labels carry no signal, so the labels here are planted
    by a random one-layer teacher of the same family: y = argmax([X | mean of
    the neighbours' X] T), T ~ N(0, 1) of shape 1204 x 41 (fp64 on the host).
    Every run starts from the same Glorot weights and sees the same sequence
    of mini-batches per (round, sub-GCN, local step).  After each round (its
    subAgg applied) the global model's loss on a fixed set of 40 clusters is
    evaluated (loss and accuracy); the mean loss of the round's local steps
    is reported too."""
    import torch
    import scipy.sparse as sp
    from gist_synth import get_config
    from paper_2102_10424_amd.step import BatchSlot, GistModel, SubGCN
    cfg = get_config("c3")
    g = cfg.make_graph()
    X = cfg.features_matrix()
    n = g.n
    deg = np.diff(g.rowptr).astype(np.float64)
    A = sp.csr_matrix((np.ones(g.nnz), g.col, g.rowptr), shape=(n, n))
    mean_nb = (A @ X.astype(np.float64)) / np.maximum(deg, 1.0)[:, None]
    T = np.random.default_rng(7).standard_normal((2 * X.shape[1], 41))
    y = np.argmax(np.concatenate([X, mean_nb], axis=1) @ T, axis=1).astype(np.int32)
    del A, mean_nb
    widths = [X.shape[1], hidden, hidden, 41]
    gh = G.GraphHandle(g)
    Xd = torch.from_numpy(X).cuda()
    sizes = np.diff(g.cluster_ptr)
    cap_n = int(np.sort(sizes)[-eval_clusters:].sum())
    cap_nnz = int(np.sort(np.diff(g.rowptr))[-cap_n:].sum()) + cap_n
    slot = BatchSlot(ctx, "sage", cap_n, cap_nnz, widths[0])
    eval_slot = BatchSlot(ctx, "sage", cap_n, cap_nnz, widths[0])
    eb = eval_slot.load(gh, np.arange(eval_clusters, dtype=np.int32) * 37 % g.n_clusters,
                        Xd, y)
    rng = np.random.default_rng(11)
    theta0 = []
    for l in range(3):
        lim = np.sqrt(6.0 / (widths[l] + widths[l + 1]))
        theta0.append([rng.uniform(-lim, lim, (widths[l], widths[l + 1])).astype(np.float32)
                       for _ in range(2)])
    batches = {}

    def batch(t, i, z):
        key = (t, i, z)
        if key not in batches:
            r = np.random.default_rng(1_000_000 + 10_000 * t + 100 * i + z)
            batches[key] = np.sort(r.choice(g.n_clusters, 20, replace=False)).astype(np.int32)
        return slot.load(gh, batches[key], Xd, y)

    full = SubGCN(ctx, "sage", widths, cap_n)
    eval_loss = torch.zeros(1, device="cuda")

    def evaluate(model):
        model.finalize()
        params = [torch.cat([model.theta[l][0], model.theta[l][1]], 0) for l in range(3)]
        logits = full.forward(eb, params)
        full.loss_and_grad(eb, eval_loss)
        acc = float((logits.argmax(dim=1).cpu() == eb.labels.cpu().long()).float().mean())
        return float(eval_loss.cpu()[0]), acc

    curves = {}
    for m in (1, 2, 4, 8):
        for policy in ("carry", "reset"):
            t0 = time.time()
            th = [[torch.from_numpy(p.copy()).cuda() for p in parts] for parts in theta0]
            model = GistModel(ctx, "sage", widths, m, th, adam=policy)
            runner = SubGCN(ctx, "sage", model.slice_widths, cap_n)
            losses = torch.empty(rounds, m, zeta, device="cuda")
            ev = [evaluate(model)]
            train = []
            for t in range(rounds):
                model.set_partitions({l: 100 + 10 * t + l for l in (1, 2)})
                model.begin_round()
                for i in range(m):
                    for z in range(zeta):
                        b = batch(t, i, z)
                        k, fresh = (t * zeta + z + 1, False) if policy == "carry" else (z + 1, z == 0)
                        runner.step(b, model.params[i], lr, adam=(model.M[i], model.V[i], k, fresh),
                                    loss_out=losses[t, i, z:z + 1])
                model.end_round()
                ev.append(evaluate(model))
                train.append(float(losses[t].mean().cpu()))
            curves[f"m{m}_{policy}"] = {"eval_loss_after_round": [round(v[0], 4) for v in ev],
                                        "eval_accuracy_after_round": [round(v[1], 4) for v in ev],
                                        "mean_local_step_loss": [round(v, 4) for v in train]}
            log(f"[curves] m={m} {policy}: eval loss {ev[0][0]:.3f} -> {ev[-1][0]:.3f}, "
                f"accuracy {ev[0][1]:.3f} -> {ev[-1][1]:.3f} ({time.time() - t0:.1f}s)")
    print(json.dumps({"loss_curves": curves, "setup": {
        "graph": "c3 SBM, 232,965 nodes, 1,500 clusters, mini-batch 20 clusters",
        "model": "3-layer GraphSAGE-mean " + "-".join(map(str, widths)),
        "labels": "planted: argmax([X | mean_nbr X] T), T ~ N(0,1) 1204 x 41, seed 7",
        "optimizer": f"Adam lr {lr}, betas (0.9, 0.999), eps 1e-8, no weight decay",
        "rounds": rounds, "zeta": zeta,
        "eval": f"global model after each round's subAgg, {eval_clusters} fixed clusters"}}),
        flush=True)


# ---------------------------------------------------------------------------
def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "the benchmark runs on exactly one GPU; --gpus must be 1"}))
        sys.exit(2)
    import torch
    from gist_synth import get_config
    from paper_2102_10424_amd import gist as G
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    ctx = G.Context(0)
    if args.copy_calib:
        copy_calibration(G, ctx)
        return
    if args.loss_curves:
        loss_curves(G, ctx, args.curve_rounds, args.curve_zeta, lr=args.curve_lr,
                    hidden=args.curve_hidden)
        return
    cfg = get_config(args.config)
    tiles = args.aggregation == "tile"
    if args.config == "c5":
        wl = LayerWorkload(cfg, ctx, args.dtype, args.d_in, clustered=tiles)
    else:
        # the SBM workloads' mini-batches are unions of clusters over block-contiguous ids
        wl = RoundWorkload(cfg, ctx, args.dtype, args.optimizer, args.adam_policy, args.zeta,
                           args.shared_batch, args.streams, args.graphs, args.lr,
                           clustered=tiles and cfg.batch_clusters is not None,
                           round_graphs=args.round_graphs)
    if args.round_graphs and args.warmup < 5:
        # the first five rounds record the round graphs (no subAgg pending,
        # then the four states of the model's alternating buffers and the
        # pipeline's four slot sets): none is recorded while timing
        log("[bench] --round-graphs: 5 warm-up rounds")
        args.warmup = 5
    ctxs = getattr(wl, "ctxs", [ctx])
    for w in range(args.warmup):
        wl.step()
        torch.cuda.synchronize()
        log(f"[bench] warmup {w + 1}/{args.warmup} done")
    pipes = getattr(wl, "pipes", [])
    for p in pipes:
        p.wait_s = 0.0
    # the timed region: no per-kernel instrumentation
    ms_step, per_step = timed_pass(wl, args.steps)
    host_wait_ms = sum(p.wait_s for p in pipes) * 1e3 / args.steps
    log(f"[bench] timed {args.steps} steps")
    # per-kernel figures from a separate pass of the same steps (eager when
    # the timed pass replayed graphs: replays carry no per-kernel events)
    prof, dropped = ({}, 0)
    psteps = args.profile_steps or args.steps
    if not args.no_profile:
        wl.use_graphs = False
        for c in ctxs:
            G.gist_profile_begin(c, 1 << 16)
        for s in range(psteps):
            wl.step()
        torch.cuda.synchronize()
        prof, dropped = merged_profile(G, ctxs)
        wl.use_graphs = args.graphs
        log(f"[bench] profiled {psteps} steps")
    extras = None
    if args.config == "c4" and not args.no_extras and not args.shared_batch:
        extras = target_figures(wl, ctx, 8, args.aggregation == "tile")
        log("[bench] target figures measured")
    wl.finish()   # a deferred subAgg (after the timed region and the profile)
    kernels = {}
    for k, v in sorted(prof.items(), key=lambda kv: -kv[1]["ms"]):
        e = dict(launches=v["launches"], ms_per_step=round(v["ms"] / psteps, 4),
                 avg_us=round(1e3 * v["ms"] / v["launches"], 2))
        if v["flops"] and is_gemm(k):
            e["tflops"] = round(v["flops"] / (v["ms"] * 1e-3) / 1e12, 2)
        if v["bytes"]:
            e["gbs"] = round(v["bytes"] / (v["ms"] * 1e-3) / 1e9, 1)
        kernels[k] = e
    roofline = None
    # the dominant device kernel; a pull of a mini-batch from pinned host
    # memory is bound by the host link, not by HBM or the matrix cores
    device = {k: v for k, v in prof.items() if not k.startswith("pull")}
    if device:
        dom, v = max(device.items(), key=lambda kv: kv[1]["ms"])
        avg_s = v["ms"] * 1e-3 / v["launches"]
        if is_gemm(dom):
            peak = PEAK["bf16" if "bf16" in dom else "f32"]
            ach = v["flops"] / v["launches"] / avg_s / 1e12
            roofline = {"kernel": dom, "bound": "mfma", "achieved": round(ach, 2),
                        "peak": peak, "unit": "TFLOP/s", "frac": round(ach / peak, 4),
                        "traffic": None, "avg_launch_us": round(avg_s * 1e6, 2),
                        "units_per_launch": round(v["flops"] / v["launches"] / 1e9, 3),
                        "unit_desc": "GFLOP per launch (2 M N K)"}
        else:
            ach = v["bytes"] / v["launches"] / avg_s / 1e9
            roofline = {"kernel": dom, "bound": "hbm", "achieved": round(ach, 1),
                        "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 4),
                        "traffic": None, "avg_launch_us": round(avg_s * 1e6, 2),
                        "units_per_launch": round(v["bytes"] / v["launches"] / 1e9, 4),
                        "unit_desc": "GB algorithmic per launch"}
    dtype_name = "bf16-in/f32-acc" if args.dtype == "bf16" else "f32"
    if roofline:
        t = recorded_traffic(roofline["kernel"], args.config, dtype_name)
        roofline["traffic"] = t
        roofline["traffic_unit"] = "bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, " \
                                   "copy-calibrated; null unless taken on these sources)"
    per_unit = wl.steps_per_unit()
    value = ms_step / per_unit
    cpu = None
    if not args.no_cpu_baseline:
        ms, what = wl.cpu_baseline()
        cpu = dict({"value": round(ms, 2), "unit": "ms", "kind": "oracle", "sample": what},
                   **cpu_info())
        if extras is not None:
            cpu["spmm_c5_ms"] = round(c5_oracle_spmm_ms(wl.graph), 1)
            cpu["spmm_c5_sample"] = ("fp64 Abar H over all 2,449,029 rows of the c5 matrix at "
                                     "width 256, SciPy CSR product on one thread, timed in full")
            log("[bench] oracle c5 aggregation timed")
            cpu["single_thread_ms"] = oracle_single_thread_ms()
            cpu["single_thread_sample"] = ("one sub-GCN step (fwd + loss + bwd + SGD), round 0, "
                                           "sub-GCN 0, fp64, of the c1 / c2 / c3 workloads, BLAS "
                                           "held to one thread")
            log("[bench] oracle single-thread steps timed")
    out = {
        "metric": METRIC, "value": round(value, 4), "unit": "ms",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "step_ms_p10_p50_p90": [round(float(x), 3) for x in np.percentile(per_step, [10, 50, 90])],
        "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": dtype_name,
        "data": "synthetic (seeded SBM / Chung-Lu / ER graphs, N(0,1) features, Glorot weights)",
        "config": dict(wl.describe(), parallelism="single GPU, m sub-GCNs back to back",
                       step="one GIST round" if per_unit > 1 else "one layer fwd+bwd",
                       value="ms per sub-GCN step (round time / (m zeta))" if per_unit > 1
                       else "ms per layer fwd+bwd"),
        "roofline": roofline, "cpu_baseline": cpu, "kernels": kernels,
        "host_batch_wait_ms_per_step": round(host_wait_ms, 3),
        "targets": extras,
        "kernels_from": (f"a separate profiled pass of {psteps} steps after the timed region "
                         "(library HIP event pairs around every launch, on its launch stream)" +
                         (", launched eagerly" if args.graphs else "")),
        "profile_dropped": dropped, "kernel_src_sha256": kernel_source_hash(),
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
