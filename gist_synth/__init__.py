"""Seeded synthetic inputs shaped like the paper's workloads.

This package produces the *inputs* of a GIST sub-GCN step and nothing else:
graphs (Erdos-Renyi, Chung-Lu power law, stochastic block model with
block-contiguous node ids standing in for METIS clusters), node features,
labels, Glorot-initialised global weights and upstream gradients.  It holds
none of the method's arithmetic (no partition, no normalisation, no layer
math), so the oracle and the HIP path can both consume it without sharing
any computation.

Every array is a pure function of an integer seed and a tuple of stream
keys (see :mod:`gist_synth.seeds`), so any process regenerates identical
bytes.  The paper's datasets (Table 5: Cora, Pubmed, Reddit, Amazon2M, ...)
are not used; these graphs only borrow their sizes and shapes.
"""

from .seeds import derive_seed, generator, philox_rows  # noqa: F401
from .graphs import Graph, erdos_renyi, chung_lu, sbm  # noqa: F401
from .tensors import (  # noqa: F401
    normal_rows, bernoulli_rows, labels_uniform, glorot_uniform, glorot_rows,
)
from .configs import CONFIGS, Config, get_config  # noqa: F401
