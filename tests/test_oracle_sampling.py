"""Pins for the oracle's generator and node sampler (CPU only)."""

import json
import os

import numpy as np
import pytest
from scipy import stats

from oracle import rng, sampling

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_splitmix64_known_answers():
    with open(os.path.join(GOLDEN, "splitmix64_kat.json")) as f:
        kat = json.load(f)
    for case in kat["cases"]:
        want = [int(x, 16) for x in case["outputs_hex"]] if "outputs_hex" in case \
            else [int(x) for x in case["outputs"]]
        got_scalar = [rng.splitmix64_scalar(case["seed"], c) for c in range(len(want))]
        got_vec = [int(v) for v in rng.splitmix64(case["seed"], np.arange(len(want)))]
        assert got_scalar == want
        assert got_vec == want


def test_splitmix64_vector_matches_scalar_on_random_counters():
    g = np.random.default_rng(5)
    seeds = [0, 1, 2 ** 63 + 17, 2 ** 64 - 1]
    ctr = g.integers(0, 2 ** 62, size=200, dtype=np.int64).astype(np.uint64)
    for s in seeds:
        vec = rng.splitmix64(s, ctr)
        for c, v in zip(ctr[:50], vec[:50]):
            assert int(v) == rng.splitmix64_scalar(s, int(c))


def test_splitmix64_keys_distinct():
    keys = rng.splitmix64(99, np.arange(1 << 18))
    assert np.unique(keys).size == keys.size


@pytest.mark.parametrize("M,s", [(1, 1), (10, 10), (1000, 1000)])
def test_sample_all_is_identity(M, s):
    assert np.array_equal(sampling.sample_nodes(M, s, 123), np.arange(M))


def test_sample_empty_and_invalid():
    assert sampling.sample_nodes(10, 0, 1).size == 0
    assert sampling.sample_nodes(0, 0, 1).size == 0
    with pytest.raises(ValueError):
        sampling.sample_nodes(5, 6, 1)


def test_sample_is_smallest_keys_bruteforce():
    # the selection rule written out with Python integers on a tiny case
    M, s, seed = 37, 9, 2024
    keys = [(rng.splitmix64_scalar(seed, m), m) for m in range(M)]
    want = sorted(m for _, m in sorted(keys)[:s])
    assert sampling.sample_nodes(M, s, seed).tolist() == want


def test_sample_properties_and_determinism():
    for seed in range(5):
        idx = sampling.sample_nodes(5000, 1234, seed)
        assert idx.dtype == np.int32 and idx.size == 1234
        assert np.all(np.diff(idx) > 0)
        assert idx.min() >= 0 and idx.max() < 5000
        assert np.array_equal(idx, sampling.sample_nodes(5000, 1234, seed))
    assert not np.array_equal(sampling.sample_nodes(5000, 1234, 0), sampling.sample_nodes(5000, 1234, 1))


def test_sample_uniform_inclusion_chi_square():
    M, s, trials = 40, 10, 4000
    counts = np.zeros(M)
    for seed in range(trials):
        counts[sampling.sample_nodes(M, s, seed)] += 1
    expected = trials * s / M
    chi2 = ((counts - expected) ** 2 / expected).sum()
    # inclusion indicators are not independent across m, but the statistic
    # is still ~chi2(M-1) up to a factor (1 - s/M) < 1; a loose bound suffices
    assert stats.chi2.sf(chi2, M - 1) > 1e-4
