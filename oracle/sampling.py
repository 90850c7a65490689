"""Nystrom node sampling (oracle side; test infrastructure only).

Sec. 2.1 forms the sampled sub-domain by drawing s nodes of the domain at
random; Algorithm 1 does this once per training sample (its node-sampling
step).  The reading used here: uniform sampling without replacement, where
candidate m receives the key splitmix64(seed, m) and the s candidates with the
smallest keys are kept.  Keys are distinct (see ``rng``), so the set is unique;
it is returned in ascending candidate order.

Pinned by: s == M gives the identity, s == 0 gives nothing, every draw is a
set of distinct in-range indices, and inclusion frequencies over many seeds
pass a chi-square uniformity test.
"""

import numpy as np

from .rng import splitmix64


def sample_nodes(M: int, s: int, seed: int) -> np.ndarray:
    """Indices of the s sampled candidates out of M, ascending, as int32."""
    if s < 0 or M < 0 or s > M:
        raise ValueError("need 0 <= s <= M")
    if s == 0:
        return np.zeros(0, dtype=np.int32)
    keys = splitmix64(seed, np.arange(M, dtype=np.uint64))
    order = np.argsort(keys, kind="stable")      # keys are distinct
    kept = np.sort(order[:s])
    return kept.astype(np.int32)
