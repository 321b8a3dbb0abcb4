"""``subGCNs``: random disjoint partition of a feature dimension into m blocks.

Paper: Section 2.1 (with its footnote example d=4, m=2 giving blocks {1,4}
and {2,3}) and Algorithm 1.  The paper asks only for a random partition into disjoint blocks of equal
size; the randomness is fixed as follows so two independent
implementations agree bit for bit:

* generator: SplitMix64 (Steele, Lea & Flood, "Fast splittable pseudorandom
  number generators", OOPSLA 2014): the state advances by the golden-ratio
  increment and each output is the state passed through the variant-13
  64-bit finaliser;
* Fisher-Yates / Durstenfeld shuffle of [0, d): for i = d-1 down to 1 draw
  j uniform on [0, i] by rejection (discard draws r >= 2^64 - (2^64 mod
  (i+1)), then j = r mod (i+1)) and swap p[i], p[j];
* block k is the slice p[k d/m : (k+1) d/m] sorted ascending; indices are
  0-based.

The categorical variant follows the masks of Appendix C.1: each index r
independently joins block j with probability 1/m (one rejection draw per r,
r ascending); block sizes are then random.
"""

MASK64 = (1 << 64) - 1
GOLDEN_GAMMA = 0x9E3779B97F4A7C15
MIX_A = 0xBF58476D1CE4E5B9
MIX_B = 0x94D049BB133111EB


class SplitMix64:
    """SplitMix64 stream: state += gamma; output = mix(state)."""

    def __init__(self, seed):
        self.state = int(seed) & MASK64

    def next(self):
        self.state = (self.state + GOLDEN_GAMMA) & MASK64
        z = self.state
        z = ((z ^ (z >> 30)) * MIX_A) & MASK64
        z = ((z ^ (z >> 27)) * MIX_B) & MASK64
        return z ^ (z >> 31)

    def below(self, bound):
        """Uniform integer on [0, bound) by rejection of the top partial range."""
        bound = int(bound)
        limit = (1 << 64) - ((1 << 64) % bound)
        while True:
            r = self.next()
            if r < limit:
                return r % bound


def shuffled(d, seed):
    """Fisher-Yates permutation of [0, d) driven by SplitMix64(seed)."""
    p = list(range(d))
    g = SplitMix64(seed)
    for i in range(d - 1, 0, -1):
        j = g.below(i + 1)
        p[i], p[j] = p[j], p[i]
    return p


def partition(d, m, seed, categorical=False):
    """Blocks D^(1..m) of [0, d) as ``(idx, offs)``.

    ``idx`` lists the blocks one after another, each ascending; block i is
    ``idx[offs[i]:offs[i+1]]``.  Equal blocks need m | d (else ValueError).
    """
    d, m = int(d), int(m)
    if m < 1 or d < 1 or m > d:
        raise ValueError("need 1 <= m <= d")
    if categorical:
        g = SplitMix64(seed)
        owner = [g.below(m) for _ in range(d)]
        blocks = [[r for r in range(d) if owner[r] == j] for j in range(m)]
    else:
        if d % m:
            raise ValueError("equal blocks need m | d")
        p = shuffled(d, seed)
        s = d // m
        blocks = [sorted(p[k * s:(k + 1) * s]) for k in range(m)]
    idx, offs = [], [0]
    for b in blocks:
        idx.extend(b)
        offs.append(len(idx))
    return idx, offs


def blocks_of(idx, offs):
    return [list(idx[offs[i]:offs[i + 1]]) for i in range(len(offs) - 1)]
