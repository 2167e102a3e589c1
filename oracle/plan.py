"""RPBH plan: uniform random permutation + Rademacher signs (test infrastructure only).

Sec. 4.4, Eq. (9): Pi_d = blkdiag(H_h D_1, ..., H_h D_{d/h}) P_pi.  The plan is
stored as a permutation array and a sign vector, drawn once per dimension and
independently of the data; h is the Hadamard block size (h | d).

The paper does not say how pi and the signs are drawn.  Reading taken: a
documented generator, SplitMix64 (Steele, Lea & Flood, "Fast splittable
pseudorandom number generators", OOPSLA 2014 -- the generator behind Java's
SplittableRandom), written here from its published definition:

    state <- state + 0x9E3779B97F4A7C15
    z <- state
    z <- (z xor (z >> 30)) * 0xBF58476D1CE4E5B9
    z <- (z xor (z >> 27)) * 0x94D049BB133111EB
    output z xor (z >> 31)                              (all mod 2^64)

The n-th output is a pure function of (seed, n), so the stream is counter based.

Draw order for plan(d, h, seed), one stream started at state = seed:
  1. perm = identity; for j = d-1 down to 1: k = uniform integer in [0, j];
     swap perm[j], perm[k]        (Fisher-Yates / Durstenfeld shuffle)
  2. for j = 0 .. d-1: sign[j] = -1 if the top bit of the next output is 1 else +1
Uniform integer in [0, n): draw u until u >= (2^64 mod n), return u mod n
(rejection makes the result exactly uniform).

Convention (reading of "permutation gather"): (P_pi x)_j = x[perm[j]], and
sign[j] multiplies the j-th post-permutation coordinate, i.e. D_j acts on the
block of positions j*h .. j*h+h-1 after the gather.
"""

from dataclasses import dataclass

import numpy as np

_MASK = (1 << 64) - 1
_GAMMA = 0x9E3779B97F4A7C15


class SplitMix64:
    """SplitMix64 from its published definition (see module docstring)."""

    def __init__(self, seed: int):
        self.state = seed & _MASK

    def next(self) -> int:
        self.state = (self.state + _GAMMA) & _MASK
        z = self.state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK
        return z ^ (z >> 31)

    def below(self, n: int) -> int:
        """Exactly uniform integer in [0, n) by rejection."""
        t = (1 << 64) % n
        while True:
            u = self.next()
            if u >= t:
                return u % n


@dataclass(frozen=True)
class Plan:
    d: int
    h: int
    perm: np.ndarray   # int64 [d], gather indices: y_j = x[perm[j]]
    sign: np.ndarray   # float64 [d] of +-1, applied after the gather


def rpbh_plan(d: int, h: int, seed: int) -> Plan:
    """Draw (pi, D) for dimension d with block size h (Eq. (9); Alg. 1, offline stage)."""
    if d < 1 or h < 1 or (h & (h - 1)) != 0 or d % h != 0:
        raise ValueError("need h a power of two dividing d")
    g = SplitMix64(seed)
    perm = list(range(d))
    for j in range(d - 1, 0, -1):
        k = g.below(j + 1)
        perm[j], perm[k] = perm[k], perm[j]
    sign = np.array([-1.0 if (g.next() >> 63) else 1.0 for _ in range(d)], dtype=np.float64)
    return Plan(d=d, h=h, perm=np.array(perm, dtype=np.int64), sign=sign)
