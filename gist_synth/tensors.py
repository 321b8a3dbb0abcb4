"""Seeded dense inputs: features, labels, initial weights, upstream gradients.

Large matrices are generated row-chunk by row-chunk from counter-based
Philox streams, in a thread pool (NumPy releases the GIL while filling), so
the result does not depend on the number of threads and any subset of rows
can be produced on its own.
"""

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from .seeds import philox_rows, generator

ROW_CHUNK = 1024


def _threads():
    return max(1, min(16, os.cpu_count() or 1))


def _chunked(shape, make, fill, rows=None, chunk=ROW_CHUNK):
    """Fill a float32 matrix chunk-wise; chunk c uses stream ``make(c)``.

    ``rows`` (optional, sorted or not) selects a subset of rows: only the
    chunks holding them are generated.
    """
    n, w = int(shape[0]), int(shape[1])
    if rows is None:
        out = np.empty((n, w), dtype=np.float32)
        nchunks = (n + chunk - 1) // chunk

        def job(c):
            a = c * chunk
            b = min(n, a + chunk)
            fill(make(c), out[a:b])

        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(job, range(nchunks)))
        return out
    rows = np.asarray(rows, dtype=np.int64)
    out = np.empty((rows.shape[0], w), dtype=np.float32)
    cids = np.unique(rows // chunk)

    def job2(c):
        a = int(c) * chunk
        b = min(n, a + chunk)
        buf = np.empty((b - a, w), dtype=np.float32)
        fill(make(int(c)), buf)
        sel = np.nonzero((rows >= a) & (rows < b))[0]
        out[sel] = buf[rows[sel] - a]

    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(job2, cids))
    return out


def normal_rows(shape, base, *keys, rows=None):
    """N(0, 1) float32 matrix of ``shape`` (or its ``rows`` subset)."""
    make = philox_rows(base, *keys)

    def fill(g, dst):
        g.standard_normal(out=dst, dtype=np.float32)

    return _chunked(shape, make, fill, rows)


def bernoulli_rows(shape, p, base, *keys, rows=None):
    """{0,1}-valued float32 matrix, each entry 1 with probability ``p``."""
    make = philox_rows(base, *keys)

    def fill(g, dst):
        dst[...] = (g.random(dst.shape, dtype=np.float32) < np.float32(p))

    return _chunked(shape, make, fill, rows)


def labels_uniform(n, classes, base, *keys):
    """int32 labels drawn uniformly from [0, classes)."""
    g = generator(base, *keys)
    return g.integers(0, classes, size=n, dtype=np.int32)


def glorot_bound(fan_in, fan_out):
    return float(np.sqrt(6.0 / (fan_in + fan_out)))


def glorot_uniform(fan_in, fan_out, base, *keys, rows=None, chunk=256):
    """Glorot-uniform float32 (fan_in x fan_out), U(-b, b), b = sqrt(6/(fan_in+fan_out)).

    Uniforms are drawn as float32 in [0, 1), mapped to [-1, 1) by the exact
    operation 2u - 1, and scaled by b (one float32 multiply).
    """
    make = philox_rows(base, *keys)
    bound = np.float32(glorot_bound(fan_in, fan_out))

    def fill(g, dst):
        g.random(out=dst, dtype=np.float32)
        dst *= np.float32(2.0)
        dst -= np.float32(1.0)
        dst *= bound

    return _chunked((fan_in, fan_out), make, fill, rows, chunk=chunk)


def glorot_rows(fan_in, fan_out, rows, base, *keys):
    """The listed rows of :func:`glorot_uniform` (same values)."""
    return glorot_uniform(fan_in, fan_out, base, *keys, rows=rows)
