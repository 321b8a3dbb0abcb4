"""Pins of the oracle's ``subGCNs`` partition (Section 2.1; Appendix C.1 masks)."""

import os

import numpy as np
import pytest

from oracle import partition as P

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line)
    return rows


def valid_partition(blocks, d, m, equal=True):
    """The defining properties: m disjoint blocks covering [0, d), equal sizes."""
    if len(blocks) != m:
        return False
    allidx = [r for b in blocks for r in b]
    if sorted(allidx) != list(range(d)):
        return False  # not a cover, or not disjoint
    if equal and any(len(b) != d // m for b in blocks):
        return False
    return all(list(b) == sorted(b) for b in blocks)


def test_splitmix64_published_outputs():
    want = [int(x, 16) for x in _read_golden("splitmix64_seed0.txt")]
    g = P.SplitMix64(0)
    assert [g.next() for _ in want] == want


def test_bounded_draw_is_uniform_and_rejects_top_range():
    g = P.SplitMix64(12345)
    for bound in (3, 7):
        cnt = np.bincount([g.below(bound) for _ in range(21000)], minlength=bound)
        exp = 21000 / bound
        chi2 = ((cnt - exp) ** 2 / exp).sum()
        assert chi2 < 30.0, (bound, cnt)
    # bound just above 2^63: about half of the raw draws are rejected, and
    # accepted values stay below the bound.
    big = (1 << 63) + 1
    vals = [g.below(big) for _ in range(200)]
    assert all(0 <= v < big for v in vals)
    raw = P.SplitMix64(99)
    acc = sum(raw.next() < (1 << 64) - ((1 << 64) % big) for _ in range(4000))
    assert 1800 < acc < 2200


def test_fisher_yates_permutations_uniform():
    # d = 4: all 24 permutations equally likely.
    counts = {}
    for s in range(24000):
        k = tuple(P.shuffled(4, s))
        counts[k] = counts.get(k, 0) + 1
    assert len(counts) == 24
    c = np.array(list(counts.values()), dtype=float)
    chi2 = ((c - 1000.0) ** 2 / 1000.0).sum()
    assert chi2 < 60.0  # 23 dof, p ~ 1e-4


@pytest.mark.parametrize("d,m", [(4, 2), (8, 4), (12, 3), (256, 2), (2048, 4),
                                 (4096, 4), (96, 96), (7, 1), (1000, 8)])
def test_partition_invariants(d, m):
    for seed in (0, 1, 2**63 + 5):
        idx, offs = P.partition(d, m, seed)
        assert offs == [i * d // m for i in range(m + 1)]
        assert valid_partition(P.blocks_of(idx, offs), d, m)


def test_mask_properties():
    # Appendix C.1: sum_j M^(j)_r = 1 and M^(j)_r M^(j')_r = 0 for j != j'.
    d, m = 64, 4
    for cat in (False, True):
        idx, offs = P.partition(d, m, 7, categorical=cat)
        M = np.zeros((m, d), dtype=int)
        for j, b in enumerate(P.blocks_of(idx, offs)):
            M[j, b] = 1
        assert (M.sum(axis=0) == 1).all()
        for j in range(m):
            for jj in range(m):
                if j != jj:
                    assert (M[j] * M[jj] == 0).all()


def test_special_cases():
    idx, offs = P.partition(10, 1, 3)
    assert idx == list(range(10)) and offs == [0, 10]
    idx, offs = P.partition(6, 6, 3)
    assert sorted(idx) == list(range(6)) and offs == list(range(7))


def test_footnote_example_is_valid_and_validator_is_not_vacuous():
    rows = _read_golden("footnote_partition.txt")
    d, m = map(int, rows[0].split())
    blocks = [[int(x) - 1 for x in r.split()] for r in rows[1:]]
    assert valid_partition(blocks, d, m)
    assert not valid_partition([[0, 3], [1, 3]], 4, 2)     # overlap
    assert not valid_partition([[0, 3], [1]], 4, 2)        # unequal / no cover
    assert not valid_partition([[3, 0], [1, 2]], 4, 2)     # unsorted
    # The oracle can produce exactly that example for some seed.
    found = any(P.blocks_of(*P.partition(4, 2, s)) == blocks for s in range(200))
    assert found


def test_membership_probability_is_one_over_m():
    # Assumption of the theory: each neuron lands in block j w.p. 1/m.
    d, m, S = 8, 4, 4000
    for cat in (False, True):
        cnt = np.zeros((d, m))
        for s in range(S):
            idx, offs = P.partition(d, m, s, categorical=cat)
            for j, b in enumerate(P.blocks_of(idx, offs)):
                cnt[b, j] += 1
        exp = S / m
        chi2 = ((cnt - exp) ** 2 / exp).sum()
        assert chi2 < 80.0, cnt  # 24 dof


def test_categorical_blocks_ascending_and_cover():
    idx, offs = P.partition(1000, 8, 11, categorical=True)
    bl = P.blocks_of(idx, offs)
    assert valid_partition(bl, 1000, 8, equal=False)
    sizes = [len(b) for b in bl]
    assert len(set(sizes)) > 1  # random sizes


def test_deterministic_and_seed_sensitive():
    a = P.partition(512, 4, 42)
    assert a == P.partition(512, 4, 42)
    assert a != P.partition(512, 4, 43)


@pytest.mark.parametrize("d,m", [(10, 3), (4, 0), (4, 5), (0, 1)])
def test_errors(d, m):
    with pytest.raises(ValueError):
        P.partition(d, m, 0)
