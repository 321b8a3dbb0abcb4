"""GPU parity of the fused subAgg + gather pass (end of one round of
Algorithm 1, start of the next): bit-exact against the oracle's subAgg of
every trained slice followed by the gather of every new slice, for both
partitioned and unpartitioned dimensions (Section 2.1), unaligned widths,
padded leading dimensions, m = 1, and either half alone.  A model-level case
checks that fused rounds leave Theta bit-identical to separate subAgg and
gather calls."""

import numpy as np
import pytest

from oracle import layers as OL
from oracle import partition as P

from gpu_util import log, to_dev, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def G():
    from paper_2102_10424_amd import gist
    return gist


@pytest.fixture(scope="module")
def ctx(G):
    return G.Context(0)


def _blocks(d, m, seed, partitioned):
    """Blocks of an equal partition (True), a categorical one ("cat": unequal,
    possibly empty blocks), one whose blocks are not in ascending order
    ("unsorted": valid, though gist_partition never returns it), or None."""
    if not partitioned:
        return None
    if partitioned == "unsorted":
        perm = np.random.default_rng(seed).permutation(d).astype(np.int32)
        s = d // m
        return [perm[i * s:(i + 1) * s] for i in range(m)]
    idx, offs = P.partition(d, m, seed, categorical=partitioned == "cat")
    return [np.asarray(idx[offs[i]:offs[i + 1]], dtype=np.int32) for i in range(m)]


def _maps(G, d, m, blocks):
    """Device (rank, offsets) of a partition given as blocks, or (None, None)."""
    if blocks is None:
        return None, None
    idx = np.concatenate(blocks).astype(np.int32)
    offs = np.cumsum([0] + [len(b) for b in blocks]).astype(np.int64)
    rank = G.gist_partition_inverse(idx, offs)
    assert np.array_equal(rank[idx], np.arange(d))
    return to_dev(rank), to_dev(offs)


class _Slices:
    def __init__(self, G, rows, cols, m, rblocks, cblocks, pad, seed):
        import torch
        # every slice is allocated for the largest block
        self.nr = rows if rblocks is None else max(len(b) for b in rblocks)
        self.nc = cols if cblocks is None else max(len(b) for b in cblocks)
        self.ld = self.nc + pad
        self.t = [torch.empty(self.nr, self.ld, device="cuda") for _ in range(m)]
        rng = np.random.default_rng(seed)
        self.host = []
        for t in self.t:
            h = rng.standard_normal((self.nr, self.ld)).astype(np.float32)
            t.copy_(torch.from_numpy(h))
            self.host.append(h)
        self.ptrs = torch.tensor([t.data_ptr() for t in self.t], dtype=torch.int64).cuda()
        self.rmaps = _maps(G, rows, m, rblocks)
        self.cmaps = _maps(G, cols, m, cblocks)
        self.rb, self.cb = rblocks, cblocks
        self.set = G.slice_set(self.rmaps[0], self.rmaps[1], self.cmaps[0], self.cmaps[1],
                               self.ptrs, self.ld)

    def rows_of(self, i):
        return None if self.rb is None else self.rb[i]

    def cols_of(self, i):
        return None if self.cb is None else self.cb[i]


CASES = [
    # rows, cols, m, rows partitioned, cols partitioned, slice pad, ldg pad
    (96, 128, 4, True, True, 0, 0),          # hidden layer
    (100, 64, 4, False, True, 0, 0),         # layer 0: input width not partitioned
    (64, 7, 2, True, False, 3, 3),           # last layer: classes not partitioned, unaligned
    (30, 30, 3, True, True, 1, 2),           # unaligned widths
    (33, 20, 1, False, False, 0, 0),         # m = 1: one sub-GCN holds all of Theta
    (40, 1500, 4, True, True, 0, 0),         # ragged last column chunk, aligned
    (4096, 4096, 8, True, True, 0, 0),       # several column chunks per row
    (50, 2052, 16, "cat", "cat", 0, 0),      # categorical: unequal (maybe empty) blocks
    (60, 44, 5, False, "cat", 1, 0),         # layer 0 with categorical columns
    (64, 1024, 4, "unsorted", "unsorted", 0, 0),  # no contiguous runs of positions
    (64, 1024, 4, True, False, 0, 0),        # last layer, aligned
    (8, 32768, 8, True, True, 0, 4),         # long rows
]


@pytest.mark.parametrize("rows,cols,m,rp,cp,spad,gpad", CASES)
@pytest.mark.parametrize("mode", ["both", "done", "next"])
def test_subagg_gather_bit_exact(G, ctx, rows, cols, m, rp, cp, spad, gpad, mode):
    import torch
    log(f"subagg_gather {rows}x{cols} m={m} rows {rp} cols {cp} mode {mode}")
    rng = np.random.default_rng(rows * 7 + cols)
    ldg = cols + gpad
    T = rng.standard_normal((rows, ldg)).astype(np.float32)
    Td = to_dev(T)
    # the two rounds draw different partitions
    done = _Slices(G, rows, cols, m, _blocks(rows, m, 11, rp), _blocks(cols, m, 12, cp), spad, 1)
    nxt = _Slices(G, rows, cols, m, _blocks(rows, m, 21, rp), _blocks(cols, m, 22, cp), spad, 2)
    G.gist_subagg_gather(ctx, Td, rows, cols, ldg, m, done.set if mode != "next" else None,
                         nxt.set if mode != "done" else None)
    torch.cuda.synchronize()
    want = T[:, :cols]
    if mode != "next":
        for i in range(m):
            nr = rows if done.rb is None else len(done.rb[i])
            nc = cols if done.cb is None else len(done.cb[i])
            want = OL.subagg(want, done.rows_of(i), done.cols_of(i), done.host[i][:nr, :nc])
    got = to_host(Td)
    assert np.array_equal(got[:, :cols].view(np.uint32), want.view(np.uint32))
    assert np.array_equal(got[:, cols:].view(np.uint32), T[:, cols:].view(np.uint32))
    for i in range(m):
        h = to_host(nxt.t[i])
        if mode != "done":
            ref = OL.gather_slice(want, nxt.rows_of(i), nxt.cols_of(i))
            a, b = ref.shape
            assert np.array_equal(h[:a, :b].view(np.uint32), ref.view(np.uint32))
            # the rest of the slice (padding, room of a smaller block) is never written
            keep = np.ones(h.shape, bool)
            keep[:a, :b] = False
            assert np.array_equal(h[keep].view(np.uint32), nxt.host[i][keep].view(np.uint32))
        else:
            assert np.array_equal(h.view(np.uint32), nxt.host[i].view(np.uint32))


def test_subagg_gather_errors(G, ctx):
    import torch
    T = torch.zeros(8, 8, device="cuda")
    ptrs = torch.zeros(2, dtype=torch.int64, device="cuda")
    unpart = G.slice_set(None, None, None, None, ptrs, 8)
    with pytest.raises(G.GistError) as e:
        G.gist_subagg_gather(ctx, T, 8, 8, 8, 2, unpart, None)
    assert e.value.status == G.GIST_E_INVAL
    with pytest.raises(G.GistError):
        G.gist_subagg_gather(ctx, T, 8, 8, 4, 1, None, unpart)   # ldg < cols
    # nothing to do
    G.gist_subagg_gather(ctx, T, 8, 8, 8, 2, None, None)
    G.gist_subagg_gather(ctx, T, 0, 8, 8, 2, unpart, unpart)


@pytest.mark.parametrize("kind", ["gcn", "sage", "gat"])
def test_fused_rounds_match_separate_calls(G, ctx, kind):
    """Three rounds of a GistModel with fused subAgg/gather and with the
    separate calls, the training replaced by a fixed change of every slice
    (different per sub-GCN, so GAT's shared output-layer attention vectors
    average distinct copies): Theta and every slice agree bit for bit."""
    import torch
    from paper_2102_10424_amd.step import GistModel
    widths, m = [40, 64, 96, 7], 4
    parts = 1 if kind == "gcn" else 2
    rng = np.random.default_rng(5)
    rows = lambda l, p: 2 if kind == "gat" and p == 1 else widths[l]
    theta0 = [[rng.standard_normal((rows(l, p), widths[l + 1])).astype(np.float32)
               for p in range(parts)] for l in range(3)]
    models = []
    for fused in (True, False):
        th = [[to_dev(t.copy()) for t in ps] for ps in theta0]
        models.append(GistModel(ctx, kind, widths, m, th, fused=fused))
    for t in range(3):
        seeds = {l: 1000 * t + l for l in (1, 2)}
        for mod in models:
            mod.set_partitions(seeds)
            mod.begin_round()
        for i in range(m):
            for l in range(3):
                a, b = models[0].params[i][l], models[1].params[i][l]
                assert torch.equal(a, b), f"round {t} sub-GCN {i} layer {l} gathered slices differ"
        for mod in models:
            for i in range(m):
                for l in range(3):
                    mod.params[i][l].mul_(-0.5).add_(float(i + 1))
            mod.end_round()
    models[0].finalize()
    torch.cuda.synchronize()
    for l in range(3):
        for p in range(parts):
            assert torch.equal(models[0].theta[l][p], models[1].theta[l][p])
        # Theta changed where some sub-GCN owned an entry
        assert not np.array_equal(to_host(models[0].theta[l][0]), theta0[l][0])


def test_fused_pass_rejects_one_table_for_both_sets(G, ctx):
    """The trained and the new slices must not share memory: both sets naming
    the same pointer table is refused before anything launches, and Theta and
    the slices are left as they were."""
    import torch
    rows, cols, m = 64, 96, 2
    blocks = _blocks(cols, m, 5, True)
    S = _Slices(G, rows, cols, m, None, blocks, 0, 9)
    Wg = torch.randn(rows, cols, device="cuda")
    before = to_host(Wg).copy()
    with pytest.raises(G.GistError) as e:
        G.gist_subagg_gather(ctx, Wg, rows, cols, cols, m, S.set, S.set)
    assert "slice table" in str(e.value)
    assert np.array_equal(to_host(Wg), before)
    for t, h in zip(S.t, S.host):
        assert np.array_equal(to_host(t), h)
