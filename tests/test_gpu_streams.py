"""Sub-GCN steps of a round spread over several HIP streams (bench.py
--streams): each stream has its own context, runner buffers and mini-batch
pipeline, starts after the fused subAgg/gather pass and joins before the
next one.  The sub-GCNs of a round touch disjoint slices and every kernel
reduces in a fixed order, so Theta and the Adam moments after the rounds
must be bitwise those of the one-stream run.  Checked on the GAT workload
(c6: per-stream pipelines, the averaged output-layer attention vectors) with
Adam moments carried through subAgg."""

import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

from gpu_util import log

pytestmark = pytest.mark.gpu


def test_two_streams_match_one_stream_bitwise():
    import torch
    import bench
    from gist_synth import get_config
    from paper_2102_10424_amd import gist as G
    ctx = G.Context(0)
    out = {}
    for ns in (1, 2):
        wl = bench.RoundWorkload(get_config("c6"), ctx, "f32", "adam", "carry", 2, False, ns)
        for _ in range(3):
            wl.step()
        wl.finish()
        torch.cuda.synchronize()
        out[ns] = [t.cpu().numpy().copy() for mats in (wl.model.theta, wl.model.Mg, wl.model.Vg)
                   for parts in mats for t in parts]
        log(f"streams={ns}: 3 rounds of 4 sub-GCNs x 2 local steps done")
        del wl
    for a, b in zip(out[1], out[2]):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
