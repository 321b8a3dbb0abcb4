"""GPU parity of the bandwidth kernels: softmax cross-entropy, slice gather
(subGCNs), subAgg scatter (bit-exact), SGD (within one fp32 ulp of the fp64
update)."""

import numpy as np
import pytest

from oracle import layers as OL
from oracle import partition as P

from gpu_util import FP32_TOL, log, relerr, to_dev, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def G():
    from paper_2102_10424_amd import gist
    return gist


@pytest.fixture(scope="module")
def ctx(G):
    return G.Context(0)


@pytest.mark.parametrize("n,C", [(1, 7), (13, 3), (1633, 47), (3106, 41), (517, 130)])
def test_softmax_xent(G, ctx, n, C):
    import torch
    log(f"xent n={n} C={C}")
    rng = np.random.default_rng(n + C)
    Z = (rng.standard_normal((n, C)) * 3).astype(np.float32)
    y = rng.integers(0, C, n).astype(np.int32)
    loss = torch.zeros(1, device="cuda")
    dZ = torch.empty(n, C, device="cuda")
    ws = torch.empty(G.gist_softmax_xent_workspace(n), dtype=torch.uint8, device="cuda")
    G.gist_softmax_xent(ctx, n, C, to_dev(Z), to_dev(y), loss, dZ, ws)
    wl, wg = OL.softmax_xent(Z, y)
    assert abs(float(to_host(loss)[0]) - wl) / abs(wl) <= FP32_TOL
    assert relerr(to_host(dZ), wg) <= FP32_TOL


@pytest.mark.parametrize("n,C,valid", [(64, 41, 50), (3200, 41, 3107), (10, 7, 0), (10, 7, 10),
                                       (10, 7, 25), (10, 7, -3)])
def test_softmax_xent_padded(G, ctx, n, C, valid):
    """A batch padded to n rows with the real count on the device: the loss is
    the oracle's over the first rows (a count outside [0, n] clamped), the
    padded rows' gradient is zero, and without padding the result is bit for
    bit the unpadded call's."""
    import torch
    log(f"xent padded n={n} C={C} valid={valid}")
    rng = np.random.default_rng(n + C + valid)
    Z = (rng.standard_normal((n, C)) * 3).astype(np.float32)
    y = rng.integers(0, C, n).astype(np.int32)
    loss = torch.full((1,), float("nan"), device="cuda")
    dZ = torch.full((n, C), float("nan"), device="cuda")
    ws = torch.empty(G.gist_softmax_xent_workspace(n), dtype=torch.uint8, device="cuda")
    nv = to_dev(np.array([valid], dtype=np.int32))
    G.gist_softmax_xent_padded(ctx, n, C, to_dev(Z), to_dev(y), nv, loss, dZ, ws)
    k = min(max(valid, 0), n)
    got_l, got_g = float(to_host(loss)[0]), to_host(dZ)
    assert np.all(got_g[k:] == 0)
    if k == 0:
        assert got_l == 0.0
        return
    wl, wg = OL.softmax_xent(Z[:k], y[:k])
    assert abs(got_l - wl) / abs(wl) <= FP32_TOL
    assert relerr(got_g[:k], wg) <= FP32_TOL
    if k == n:
        loss2 = torch.zeros(1, device="cuda")
        dZ2 = torch.empty(n, C, device="cuda")
        G.gist_softmax_xent(ctx, n, C, to_dev(Z), to_dev(y), loss2, dZ2, ws)
        assert torch.equal(loss, loss2) and torch.equal(dZ, dZ2)


def test_copy_pulls_from_pinned_and_device_memory(G, ctx):
    """gist_copy: every byte count (aligned, unaligned, tails), from pinned
    host memory and from device memory, and the event it records."""
    import torch
    src_h = torch.randint(0, 255, (100003,), dtype=torch.uint8).pin_memory()
    src_d = src_h.cuda()
    ev = G.Event()
    for nbytes in (0, 1, 15, 16, 17, 4096, 100000, 100003):
        for src, off in ((src_h, 0), (src_h, 3), (src_d, 0), (src_d, 5)):
            if off + nbytes > src.numel():
                continue
            dst = torch.zeros(100016, dtype=torch.uint8, device="cuda")
            G.gist_copy(ctx, dst, src.data_ptr() + off, nbytes, ev)
            ev.synchronize()
            got = dst.cpu().numpy()
            want = src_h.numpy()[off:off + nbytes]
            assert np.array_equal(got[:nbytes], want), (nbytes, off)
            assert not got[nbytes:].any()


def test_softmax_bad_label_reports_nan(G, ctx):
    import torch
    Z = torch.zeros(4, 3, device="cuda")
    y = to_dev(np.array([0, 1, 3, 2], dtype=np.int32))
    loss = torch.zeros(1, device="cuda")
    dZ = torch.empty(4, 3, device="cuda")
    ws = torch.empty(G.gist_softmax_xent_workspace(4), dtype=torch.uint8, device="cuda")
    G.gist_softmax_xent(ctx, 4, 3, Z, y, loss, dZ, ws)
    assert np.isnan(to_host(loss)[0])


@pytest.mark.parametrize("dr,dc,m", [(100, 32768, 8), (4096, 4096, 4), (256, 7, 2),
                                     (1433, 256, 2)])
def test_gather_scatter_bit_exact(G, ctx, dr, dc, m):
    import torch
    log(f"gather/scatter {dr}x{dc} m={m}")
    rng = np.random.default_rng(dr)
    T = rng.standard_normal((dr, dc)).astype(np.float32)
    Td = to_dev(T)
    ri, ro = P.partition(dr, m, 1) if dr % m == 0 and dr > 7 else (None, None)
    ci, co = P.partition(dc, m, 2) if dc % m == 0 and dc > 7 else (None, None)
    for i in range(m):
        rows = None if ri is None else np.asarray(ri[ro[i]:ro[i + 1]], dtype=np.int32)
        cols = None if ci is None else np.asarray(ci[co[i]:co[i + 1]], dtype=np.int32)
        nr = dr if rows is None else len(rows)
        nc = dc if cols is None else len(cols)
        S = torch.empty(nr, nc, device="cuda")
        rd = None if rows is None else to_dev(rows)
        cd = None if cols is None else to_dev(cols)
        G.gist_gather_slice(ctx, Td, dc, rd, nr, cd, nc, S, nc)
        want = OL.gather_slice(T, rows, cols)
        got = to_host(S)
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
        # train-like change, then subAgg it back
        S.mul_(-2.0)
        G.gist_subagg(ctx, Td, dc, rd, nr, cd, nc, S, nc)
        T = OL.subagg(T, rows, cols, -2.0 * want)
    assert np.array_equal(to_host(Td).view(np.uint32), T.view(np.uint32))


def test_subagg_check_finite(G, ctx):
    import torch
    Tg = torch.zeros(8, 8, device="cuda")
    S = torch.ones(2, 8, device="cuda")
    S[1, 3] = float("nan")
    rows = to_dev(np.array([1, 5], dtype=np.int32))
    with pytest.raises(G.GistError) as e:
        G.gist_subagg(ctx, Tg, 8, rows, 2, None, 8, S, 8, G.GIST_SUBAGG_CHECK_FINITE)
    assert e.value.status == G.GIST_E_NONFINITE
    assert float(to_host(Tg).max()) == 0.0  # nothing written
    S[1, 3] = 2.0
    G.gist_subagg(ctx, Tg, 8, rows, 2, None, 8, S, 8, G.GIST_SUBAGG_CHECK_FINITE)
    h = to_host(Tg)
    assert h[5, 3] == 2.0 and h[1].sum() == 8.0 and h[0].sum() == 0.0


@pytest.mark.parametrize("n", [1, 1000, 4096 * 4096 + 3])
def test_sgd_within_one_ulp(G, ctx, n):
    log(f"sgd n={n}")
    rng = np.random.default_rng(n % 1000)
    W = rng.standard_normal(n).astype(np.float32)
    dW = rng.standard_normal(n).astype(np.float32)
    lr = 0.0375
    Wd = to_dev(W)
    G.gist_sgd_update(ctx, Wd, to_dev(dW), n, lr)
    got = to_host(Wd)
    want = OL.sgd(W, dW, np.float32(lr)).astype(np.float32)
    ulp = np.abs(got.view(np.int32).astype(np.int64) - want.view(np.int32).astype(np.int64))
    assert ulp.max() <= 1
