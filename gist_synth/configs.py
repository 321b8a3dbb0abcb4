"""The five workloads, as seeded synthetic inputs.

Sizes follow the paper's datasets (Table 5) and experiments (Tables 1-3):

* ``c1`` 2-layer GCN, m=2, Erdos-Renyi N=2,000 (mean degree 4), 1,433 binary
  features, hidden 256, 7 classes (a Cora-sized graph).
* ``c2`` 3-layer GCN, m=4, Chung-Lu power law (exponent 2.5) N=20,000,
  mean degree 5, 500 features, hidden 2,048, 3 classes (Pubmed-sized).
* ``c3`` 4-layer GraphSAGE-mean, m=4, SBM N=232,965 in 1,500 blocks, mean
  degree 50 (90% intra-block), 602 features, hidden 4,096, 41 classes;
  mini-batch = 20 random blocks (Reddit-sized).
* ``c4`` 4-layer GraphSAGE-mean, m=8, SBM N=2,449,029 in 15,000 blocks,
  ~61.9M edges, 100 features, hidden 32,768, 47 classes; mini-batch = 10
  random blocks (Amazon2M-sized, the ultra-wide model of Table 3).
* ``c5`` one GCN layer over the whole c4 graph, input slice d_in in
  {100, 256, 512}, output = one 256-wide slice of a 2,048-wide layer (m=8).
* ``c6`` 3-layer GAT, m=4, on the c3 graph (same graph, features, labels
  and 20-block mini-batches), hidden 256 split into 4 x 64, 41 classes: the
  256-dimensional GAT the paper trains on Reddit (Table 2).
* ``c7`` GIST with LADIES layer sampling (Section 5.4, Table 4): 2-layer GCN
  602-256-41, m=4, on the c3 graph; a mini-batch is 512 output nodes drawn
  uniformly and 512 LADIES draws per layer.

Seeds: config ``k`` uses base seed 100 + k; every array is a named stream of
that base (see :mod:`gist_synth.seeds`).
"""

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

from . import graphs as _g
from . import tensors as _t
from .seeds import (STREAM_FEATURES, STREAM_LABELS, STREAM_THETA,
                    STREAM_PARTITION, STREAM_MINIBATCH, STREAM_UPSTREAM, STREAM_LADIES,
                    derive_seed, generator)


@dataclass
class Config:
    name: str
    kind: str                 # "gcn" | "sage" | "gat"
    widths: List[int]         # d_0 .. d_L (global model)
    m: int                    # number of sub-GCNs
    graph: dict               # generator name + parameters
    features: str             # "bernoulli" | "normal"
    batch_clusters: Optional[int] = None   # None: full graph
    feature_p: float = 0.0
    extra: dict = field(default_factory=dict)

    @property
    def index(self):
        return int(self.name[1:])

    @property
    def seed(self):
        return 100 + self.index

    @property
    def L(self):
        return len(self.widths) - 1

    @property
    def classes(self):
        return self.widths[-1]

    def slice_widths(self):
        """Sub-GCN widths s_0..s_L: hidden widths divided by m, d_0 and d_L kept."""
        s = list(self.widths)
        for l in range(1, self.L):
            s[l] = self.widths[l] // self.m
        return s

    # ---- inputs -------------------------------------------------------
    def make_graph(self):
        g = dict(self.graph)
        kind = g.pop("kind")
        if kind == "er":
            return _g.erdos_renyi(g["n"], g["edges"], self.seed)
        if kind == "chung_lu":
            return _g.chung_lu(g["n"], g["gamma"], g["mean_degree"], self.seed)
        if kind == "sbm":
            return _g.sbm(g["n"], g["blocks"], g["mean_degree"], g["intra"],
                          self._graph_seed())
        raise ValueError(kind)

    def _graph_seed(self):
        # c4 and c5 share one graph.
        return self.extra.get("graph_seed", self.seed)

    @property
    def n_nodes(self):
        return int(self.graph["n"])

    def features_matrix(self, rows=None):
        n, d = self.n_nodes, self.widths[0]
        base = self._graph_seed()
        if self.features == "bernoulli":
            return _t.bernoulli_rows((n, d), self.feature_p, base,
                                     STREAM_FEATURES, d, rows=rows)
        return _t.normal_rows((n, d), base, STREAM_FEATURES, d, rows=rows)

    def labels(self):
        return _t.labels_uniform(self.n_nodes, self.classes, self._graph_seed(),
                                 STREAM_LABELS, self.classes)

    def theta(self, layer, part=0, rows=None):
        """Global weight Theta_layer (d_l x d_{l+1}); SAGE part 0 = W_self,
        1 = W_neigh; GAT part 1 = the attention vectors [a_src; a_dst]
        (2 x d_{l+1}, Glorot-uniform over that shape)."""
        fi, fo = self.widths[layer], self.widths[layer + 1]
        if self.kind == "gat" and part == 1:
            fi = 2
        return _t.glorot_uniform(fi, fo, self.seed, STREAM_THETA, layer, part,
                                 rows=rows)

    def n_parts(self):
        return 1 if self.kind == "gcn" else 2

    def partition_seed(self, t, layer):
        """Seed of the feature partition of hidden dim ``layer`` in round ``t``."""
        return derive_seed(self.seed, STREAM_PARTITION, t, layer)

    def minibatch(self, t, i, z=0):
        """Cluster ids of sub-GCN ``i``'s mini-batch at round ``t``, local step ``z``.

        Returns ``None`` for full-graph configs.
        """
        if self.batch_clusters is None:
            return None
        g = generator(self.seed, STREAM_MINIBATCH, t, i, z)
        c = int(self.graph["blocks"])
        return np.sort(g.choice(c, size=self.batch_clusters, replace=False)
                       ).astype(np.int32)

    @property
    def ladies(self):
        """LADIES sizes dict(batch=b, samples=s), or None (cluster mini-batches)."""
        return self.extra.get("ladies")

    def ladies_batch(self, t, i, z=0):
        """Output nodes of sub-GCN ``i``'s LADIES mini-batch at round ``t``, step
        ``z``: ``batch`` distinct nodes drawn uniformly, ascending."""
        g = generator(self.seed, STREAM_MINIBATCH, t, i, z)
        return np.sort(g.choice(self.n_nodes, size=self.ladies["batch"], replace=False)
                       ).astype(np.int32)

    def ladies_seed(self, t, i, z=0):
        """Seed of the LADIES draws of that mini-batch."""
        return derive_seed(self.seed, STREAM_LADIES, t, i, z)

    def upstream(self, n, w, rows=None):
        """Seeded N(0,1) upstream gradient dH' (n x w) for single-layer workloads."""
        return _t.normal_rows((n, w), self.seed, STREAM_UPSTREAM, w, rows=rows)


_SBM_C4 = dict(kind="sbm", n=2_449_029, blocks=15_000, mean_degree=50.55,
               intra=0.9)

CONFIGS = {
    "c1": Config("c1", "gcn", [1433, 256, 7], 2,
                 dict(kind="er", n=2000, edges=4000), "bernoulli",
                 feature_p=0.013),
    "c2": Config("c2", "gcn", [500, 2048, 2048, 3], 4,
                 dict(kind="chung_lu", n=20_000, gamma=2.5, mean_degree=5.0),
                 "normal"),
    "c3": Config("c3", "sage", [602, 4096, 4096, 4096, 41], 4,
                 dict(kind="sbm", n=232_965, blocks=1500, mean_degree=50.0,
                      intra=0.9), "normal", batch_clusters=20),
    "c4": Config("c4", "sage", [100, 32768, 32768, 32768, 47], 8,
                 dict(_SBM_C4), "normal", batch_clusters=10),
    # c5: widths = [d_in, 2048]; the step uses output slice 0 of the m=8 split.
    "c5": Config("c5", "gcn", [256, 2048], 8, dict(_SBM_C4), "normal",
                 extra=dict(graph_seed=104, d_in_sweep=(100, 256, 512))),
    # c6: the c3 graph (graph_seed 103) with a GAT model.
    "c6": Config("c6", "gat", [602, 256, 256, 41], 4,
                 dict(kind="sbm", n=232_965, blocks=1500, mean_degree=50.0,
                      intra=0.9), "normal", batch_clusters=20,
                 extra=dict(graph_seed=103)),
    # c7: the c3 graph with a 2-layer GCN trained on LADIES mini-batches.
    "c7": Config("c7", "gcn", [602, 256, 41], 4,
                 dict(kind="sbm", n=232_965, blocks=1500, mean_degree=50.0,
                      intra=0.9), "normal",
                 extra=dict(graph_seed=103, ladies=dict(batch=512, samples=512))),
}


def get_config(name, **overrides):
    import copy
    cfg = copy.deepcopy(CONFIGS[name])
    for k, v in overrides.items():
        setattr(cfg, k, v)
    return cfg
