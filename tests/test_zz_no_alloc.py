"""The no-allocation loss entry point (gist_softmax_xent_noalloc) against
gist_softmax_xent with a caller workspace, through the C ABI: two calls in a
row on the same device, the second with fewer rows (the shared per-device
buffer keeps the first call's partial sums, which must not leak into the
second), bitwise equal loss and gradient; the row limit is an error before
any launch.  Runs alone in a fresh process and after the other tests."""

import numpy as np
import pytest

from gpu_util import log, to_dev, to_host

pytestmark = pytest.mark.gpu


def test_softmax_xent_noalloc_matches_workspace_call():
    import torch
    from paper_2102_10424_amd import gist as G
    ctx = G.Context(0)
    rng = np.random.default_rng(17)
    for n, C in ((70001, 47), (1633, 41), (3, 7), (0, 5)):
        log(f"noalloc loss n={n} C={C}")
        Z = to_dev((rng.standard_normal((max(n, 1), C)) * 3).astype(np.float32))[:n]
        y = to_dev(rng.integers(0, C, max(n, 1)).astype(np.int32))[:n]
        loss_a = torch.full((1,), float("nan"), device="cuda")
        loss_b = torch.full((1,), float("nan"), device="cuda")
        dz_a = torch.full((max(n, 1), C), float("nan"), device="cuda")[:n]
        dz_b = torch.full((max(n, 1), C), float("nan"), device="cuda")[:n]
        ws = torch.empty(G.gist_softmax_xent_workspace(n), dtype=torch.uint8, device="cuda")
        G.gist_softmax_xent(ctx, n, C, Z, y, loss_a, dz_a, ws)
        G.gist_softmax_xent_noalloc(ctx, n, C, Z, y, loss_b, dz_b)
        la, lb = to_host(loss_a), to_host(loss_b)
        assert np.array_equal(la, lb), (n, la, lb)
        assert np.array_equal(to_host(dz_a), to_host(dz_b))
        if n == 0:
            assert lb[0] == 0.0
        else:   # and the loss is the mean cross-entropy of these logits
            z = to_host(Z).astype(np.float64)
            yy = to_host(y)
            m = z.max(axis=1, keepdims=True)
            lse = m[:, 0] + np.log(np.exp(z - m).sum(axis=1))
            want = np.mean(lse - z[np.arange(n), yy])
            assert abs(lb[0] - want) <= 1e-5 * abs(want)
    with pytest.raises(G.GistError) as e:
        G.gist_softmax_xent_noalloc(ctx, G.GIST_NOALLOC_LOSS_MAX_ROWS + 1, 2, Z, y, loss_b, dz_b)
    assert e.value.status == G.GIST_E_INVAL
