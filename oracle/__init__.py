"""Plain fp64 CPU oracle for the GIST sub-GCN training step.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
library (no kernels, headers, helpers or tables) and does not import it.

What it computes, each function citing the passage it follows (paper:
"GIST: Distributed Training for Large-Scale Graph Convolutional Networks"):

* :mod:`oracle.partition` -- ``subGCNs`` feature partition (Section 2.1 and
  its footnote; Algorithm 1), SplitMix64 + Fisher-Yates, plus the
  categorical-mask variant of the theory appendix (Appendix C.1).
* :mod:`oracle.minibatch` -- ``Cluster`` mini-batch: union of clusters,
  induced subgraph, normalised aggregation matrix (Section 2.2 for the
  mini-batch; eq. (1) for the self-looped degree-normalised matrix;
  eq. "Aggregation Matrix" of Appendix C.2 for the theory form).
* :mod:`oracle.layers` -- the sub-GCN layer forward and backward (eq. (1),
  eq. (2)), the GraphSAGE-mean layer, softmax cross-entropy, SGD
  (Section 2.2), slice gather (Section 2.1) and ``subAgg`` (Section 2.2).
* :mod:`oracle.gist` -- one sub-GCN training step and one GIST round
  (Algorithm 1) composed from the above, and the whole loop of Algorithm 1
  trained with Adam (the optimizer of the paper's experiments).
* :mod:`oracle.optim` -- Adam (Kingma & Ba 2015, their Algorithm 1).
* :mod:`oracle.gat` -- the graph attention layer GIST is also applied to
  (Section 2.3; Table 2), single head as Velickovic et al. 2018 define it.
* :mod:`oracle.ladies` -- LADIES layer-wise sampled mini-batches, the node
  sampling GIST is combined with in place of graph partitioning
  (Section 5.4, Appendix A.6), as Zou et al. 2019 define it; the GCN layers
  of :mod:`oracle.layers` take its rectangular per-layer matrices.

Floating point is fp64 throughout; fp32 inputs are widened exactly.  The
matrices of the normalised adjacency are the one place where fp32 is part
of the definition: the values are computed in fp64 and rounded once to fp32
(round-to-nearest-even), which is what the library stores.

Every function here is pinned by ``tests/test_oracle_*.py`` against facts
the paper and the mathematics fix (published generator outputs, mask
properties, spectra, closed-form gradients, finite differences, the
two-layer sum decomposition, an independent Adam implementation); none is
"parity unpinned".
"""

from . import partition, minibatch, layers, gist, optim, gat, ladies  # noqa: F401
