"""Seed derivation for the synthetic inputs.

A stream is named by a base seed and a tuple of small integer keys (for
example ``(base, STREAM_THETA, layer, part)``).  ``derive_seed`` hashes them
with NumPy's SeedSequence into one 64-bit value; ``philox_rows`` builds a
counter-based Philox stream per row so that any subset of rows of a large
matrix can be regenerated without producing the rest.
"""

import numpy as np

# Stream identifiers (stable: changing one changes every generated input).
STREAM_GRAPH = 1
STREAM_FEATURES = 2
STREAM_LABELS = 3
STREAM_THETA = 4
STREAM_PARTITION = 5
STREAM_MINIBATCH = 6
STREAM_UPSTREAM = 7
STREAM_LADIES = 8


def derive_seed(base, *keys):
    """64-bit seed for the stream ``(base, *keys)`` (SeedSequence hash)."""
    ss = np.random.SeedSequence([int(base) & 0xFFFFFFFF, *[int(k) for k in keys]])
    return int(ss.generate_state(1, dtype=np.uint64)[0])


def generator(base, *keys):
    """A PCG64 ``numpy.random.Generator`` for the stream ``(base, *keys)``."""
    return np.random.Generator(np.random.PCG64(derive_seed(base, *keys)))


def philox_rows(base, *keys):
    """Return ``make(row) -> Generator``: one independent Philox stream per row.

    The Philox key is derived from the stream name, and the row index is the
    second word of the 256-bit counter, so rows never overlap as long as a
    row draws fewer than 2**64 blocks.
    """
    key = derive_seed(base, *keys)

    def make(row):
        return np.random.Generator(
            np.random.Philox(key=key, counter=[0, int(row), 0, 0]))

    return make
