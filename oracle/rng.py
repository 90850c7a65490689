"""SplitMix64 counter-based generator (oracle side; test infrastructure only).

The paper draws nodes and edges "randomly" (Sec. 2.1; Algorithm 1, node and
edge sampling steps) without naming a generator.  To let a GPU reproduce the
draws exactly, every random number is the SplitMix64 output for a counter:

    state_c = seed + (c + 1) * 0x9E3779B97F4A7C15        (mod 2**64)
    z = state_c
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9              (mod 2**64)
    z = (z ^ (z >> 27)) * 0x94D049BB133111EB              (mod 2**64)
    out = z ^ (z >> 31)

which is the (c+1)-th output of SplitMix64 seeded with ``seed`` (Steele, Lea
and Flood, "Fast splittable pseudorandom number generators", OOPSLA 2014; the
finaliser constants are Stafford's "Mix13").  The finaliser is a bijection of
64-bit words and the state map is injective in c, so keys of distinct
counters never collide.

Pinned by: published known-answer outputs (seed 0 and seed 1234567), and the
bijection property on random words.
"""

import numpy as np

GOLDEN = 0x9E3779B97F4A7C15
MUL1 = 0xBF58476D1CE4E5B9
MUL2 = 0x94D049BB133111EB
_MASK = (1 << 64) - 1


def splitmix64_scalar(seed: int, counter: int) -> int:
    """Key for one counter, in Python integers (slow, obviously correct)."""
    z = (seed + (counter + 1) * GOLDEN) & _MASK
    z = ((z ^ (z >> 30)) * MUL1) & _MASK
    z = ((z ^ (z >> 27)) * MUL2) & _MASK
    return z ^ (z >> 31)


def splitmix64(seed: int, counters: np.ndarray) -> np.ndarray:
    """Vectorised keys for an array of counters (uint64 wrap-around arithmetic)."""
    c = np.asarray(counters, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = np.uint64(seed & _MASK) + (c + np.uint64(1)) * np.uint64(GOLDEN)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(MUL1)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(MUL2)
        z = z ^ (z >> np.uint64(31))
    return z
