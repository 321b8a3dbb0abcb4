"""Whole GIST rounds replayed from one HIP graph each (``RoundReplayer``)
against rounds whose sub-GCN steps are replayed one by one.

Both run the benchmark's own workloads at their real shapes (c7: 2-layer GCN
on LADIES batches of the 232,965-node graph; c6: 3-layer GAT on 20-cluster
batches of the same graph), from the same initial model and the same
mini-batch and partition seeds, for seven rounds: the first five record the
round graphs (no pending subAgg, then the four states of the model's
alternating buffers and the pipeline's four slot sets), the last two replay
them.  The
round graph launches the same kernels on the same data in the same order as
the step replays plus the eager fused subAgg + gather, so the global model
after the final subAgg must agree bit for bit.
"""

import pytest

from gpu_util import log

pytestmark = pytest.mark.gpu

ROUNDS = 7


@pytest.mark.parametrize("config", ["c7", "c6"])
def test_round_replays_match_step_replays(config):
    import torch
    import bench
    from gist_synth import get_config
    from paper_2102_10424_amd import gist as G
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    ctx = G.Context(0)
    cfg = get_config(config)
    thetas = []
    for round_graphs in (False, True):
        log(f"{config}: {ROUNDS} rounds, round graphs {round_graphs}")
        wl = bench.RoundWorkload(cfg, ctx, "f32", graphs=True, lr=0.01, clustered=True,
                                 round_graphs=round_graphs)
        for _ in range(ROUNDS):
            wl.step()
        wl.finish()
        torch.cuda.synchronize()
        if round_graphs:
            rr = wl.round_replayer
            log(f"  recorded {len(rr.replays)} round graphs, {rr.stepwise_rounds} rounds "
                "step by step")
            assert len(rr.replays) + rr.stepwise_rounds >= 1
        thetas.append([[t.cpu().numpy().copy() for t in parts] for parts in wl.model.theta])
        del wl
        torch.cuda.synchronize()
    for l, (a, b) in enumerate(zip(*thetas)):
        for p, (x, y) in enumerate(zip(a, b)):
            assert x.tobytes() == y.tobytes(), (config, l, p)


def test_round_with_a_batch_beyond_the_fixed_layout_runs_step_by_step(monkeypatch):
    """A LADIES batch with more entries than the fixed layout holds is run
    eagerly at its own shape; a round holding one runs step by step (the
    fused subAgg + gather eagerly, then each sub-GCN's step replayed or, for
    that batch, eager).  Such batches are forced here from the host (every
    batch whose first layer has a multiple of 3 entries reports that it does
    not fit), identically in both runs, so the rounds with round replays must
    still match per-step replays bit for bit."""
    import torch
    import bench
    from gist_synth import get_config
    from paper_2102_10424_amd import gist as G
    from paper_2102_10424_amd import step as S
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    real = S.LadiesSlot.fits_fixed
    monkeypatch.setattr(S.LadiesSlot, "fits_fixed",
                        lambda self: real(self) and self.built[1][0][2] % 3 != 0)
    ctx = G.Context(0)
    cfg = get_config("c7")
    thetas = []
    for round_graphs in (False, True):
        wl = bench.RoundWorkload(cfg, ctx, "f32", graphs=True, lr=0.01,
                                 round_graphs=round_graphs)
        for _ in range(ROUNDS):
            wl.step()
        wl.finish()
        torch.cuda.synchronize()
        if round_graphs:
            rr = wl.round_replayer
            log(f"c7 forced: {len(rr.replays)} round graphs, {rr.stepwise_rounds} rounds "
                "step by step")
            assert rr.stepwise_rounds >= 1
        thetas.append([[t.cpu().numpy().copy() for t in parts] for parts in wl.model.theta])
        del wl
        torch.cuda.synchronize()
    for l, (a, b) in enumerate(zip(*thetas)):
        for p, (x, y) in enumerate(zip(a, b)):
            assert x.tobytes() == y.tobytes(), (l, p)
