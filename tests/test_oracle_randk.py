"""Pins for the oracle's GlobalRandK selection (Sec. 3.3-3.4): K coordinates
chosen uniformly at random, the same for every worker.

A uniformly random K-subset has inclusion probability K/d for every
coordinate and K(K-1)/(d(d-1)) for every pair; the keys come from the Philox
blocks pinned in test_oracle_philox.py.
"""
import math

import numpy as np
import pytest


def test_sorted_distinct_in_range(orc):
    for d, K, seed in ((1, 1, 0), (10, 10, 3), (1000, 1, 9), (5000, 123, 4), (70_000, 10_000, 2)):
        s = orc.randk_select(d, K, seed).astype(np.int64)
        assert s.size == K and np.all(np.diff(s) > 0) and s[0] >= 0 and s[-1] < d


def test_keys_use_each_word_of_a_block_once(orc):
    seed = 0xABCDEF0123456789
    for q in (0, 7, 1 << 20):
        hi, lo = orc.randk_keys(seed, 4 * q, 4)
        key = [seed & 0xFFFFFFFF, seed >> 32]
        assert list(hi) == list(orc.philox([q, 0, 0, 2], key))
        assert list(lo) == list(orc.philox([q, 0, 0, 3], key))


def test_k_equal_d_and_k_one():
    from oracle import oracle as O

    assert list(O.randk_select(17, 17, 5)) == list(range(17))
    hi, lo = O.randk_keys(5, 0, 300)
    key = (hi.astype(np.uint64) << np.uint64(32)) | lo.astype(np.uint64)
    assert O.randk_select(300, 1, 5)[0] == int(np.argmin(key))


def test_inclusion_probabilities_are_uniform(orc):
    d, K, seeds = 40, 7, 6000
    count = np.zeros(d)
    pair = 0
    for seed in range(seeds):
        s = orc.randk_select(d, K, seed)
        count[s] += 1
        pair += (3 in s) and (17 in s)
    p = K / d
    sd = math.sqrt(seeds * p * (1 - p))
    assert np.max(np.abs(count - seeds * p)) < 5 * sd
    chi2 = np.sum((count - seeds * p) ** 2 / (seeds * p))
    assert chi2 < 100  # ~39 degrees of freedom (the total is fixed)
    pp = K * (K - 1) / (d * (d - 1))
    assert abs(pair - seeds * pp) < 6 * math.sqrt(seeds * pp)


def test_seeds_give_different_sets(orc):
    a = orc.randk_select(100_000, 1000, 1)
    b = orc.randk_select(100_000, 1000, 2)
    assert len(np.intersect1d(a, b)) < 60  # ~10 expected


def test_randk_step_is_quantiser_on_the_sampled_coordinates(orc):
    """Zero off the sample; on it, Algorithm 1 applied to the gathered
    sub-vectors (its own max norm over the K coordinates)."""
    rng = np.random.default_rng(3)
    M, d, K = 3, 5000, 300
    g = (rng.normal(size=(M, d)) * 1e-2).astype(np.float32)
    r = orc.randk_pipeline(g, K, [127.0], seed=11)
    sel = r["sel"].astype(np.int64)
    off = np.ones(d, dtype=bool)
    off[sel] = False
    assert not r["full"][off].any()
    sub = g[:, sel]
    assert r["W"] == orc.shared_scale(sub)[0]
    direct = orc.pipeline(sub, [127.0], 11)
    assert np.array_equal(r["full"][sel], direct["out"])


def test_randk_expectation_is_k_over_d_of_the_mean(orc):
    """E[ghat] = (K/d) * mean_m g^m: the sample is uniform and the quantiser
    unbiased; the paper applies no d/K correction."""
    rng = np.random.default_rng(5)
    M, d, K = 2, 60, 15
    g = rng.uniform(0.5, 1.0, size=(M, d)).astype(np.float32)
    seeds = 3000
    acc = np.zeros(d)
    for seed in range(seeds):
        acc += orc.randk_pipeline(g, K, [7.0], seed=seed)["full"]
    mean = acc / seeds
    target = (K / d) * g.astype(np.float64).mean(axis=0)
    # per-coordinate sd of one draw <= max|ghat| * sqrt(p(1-p)) + quantisation noise
    W = float(np.sqrt((g.astype(np.float64) ** 2).sum(axis=1)).max())
    sd = (np.abs(g).max() + W / 7.0) * math.sqrt((K / d) * (1 - K / d)) / math.sqrt(seeds)
    assert np.max(np.abs(mean - target)) < 6 * sd
