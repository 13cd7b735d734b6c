"""Pins for the oracle's stochastic quantiser, Eq. (7)-(8) and Eq. (10)/(12).

What the paper fixes: the code is sign(v_i) * (l or l+1) with l the level
below a * s (Eq. (8)); it is l+1 with probability p = a s - l, so the
quantiser is unbiased and its variance is sum_i (W/s*_i)^2 p_i (1 - p_i),
bounded by (1 + min(n/s^2, sqrt(n)/s)) W^2 (Lemma 1, Lemma 2, Appendix C/E).
A zero vector maps to zero.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import exact

HERE = os.path.dirname(os.path.abspath(__file__))
GOLD = json.load(open(os.path.join(HERE, "golden", "worked_examples.json")))


def _x_and_t(v, W, scales, idx=None):
    """The oracle's grid position x and 32-bit threshold, recomputed in numpy."""
    s = np.asarray(scales, dtype=np.float32)
    k = np.zeros(v.size, dtype=np.int64) if idx is None else np.minimum(idx, s.size - 1)
    inv = (s / np.float32(W)).astype(np.float32)
    x = np.minimum(np.abs(v).astype(np.float32) * inv[k], s[0]).astype(np.float32)
    l = np.floor(x)
    p = (x - l).astype(np.float32)
    t = (p.astype(np.float64) * 2.0 ** 32).astype(np.uint64)
    return x, l.astype(np.int64), t


def test_example_A_deterministic_levels(orc):
    ex = GOLD["A"]
    g = np.array(ex["rows"], dtype=np.float32)
    W, _ = orc.shared_scale(g)
    assert W == np.float32(ex["W"])
    for seed in range(64):
        codes = orc.quantize(g[0], W, ex["scales"], seed)
        assert list(codes) == ex["codes"][0]


def test_example_B_top_level(orc):
    ex = GOLD["B"]
    g = np.array(ex["rows"], dtype=np.float32)
    W, _ = orc.shared_scale(g)
    for seed in range(64):
        assert list(orc.quantize(g[0], W, ex["scales"], seed)) == ex["codes"][0]


def test_example_C_fair_coin(orc):
    ex = GOLD["C"]
    v = np.array(ex["rows"][0], dtype=np.float32)
    n_seeds = 4096
    up = 0
    for seed in range(n_seeds):
        c = orc.quantize(v, ex["W"], ex["scales"], seed)
        assert set(np.abs(c)) <= {1, 2}
        assert np.all(np.sign(c) == np.sign(v))
        up += int((np.abs(c) == 2).sum())
    n = n_seeds * v.size
    assert abs(up / n - ex["p_up"]) < 6 * math.sqrt(0.25 / n)


def test_example_D_shared_threshold(orc):
    ex = GOLD["D"]
    g = np.array(ex["shared"]["rows"], dtype=np.float32)
    idx = orc.scale_index_shared(g, ex["W"], ex["scales"])
    x, l, t = _x_and_t(g[0], ex["W"], ex["scales"], idx)
    assert l[0] == ex["shared"]["worker0_l"] and t[0] == ex["shared"]["worker0_threshold"]
    up = 0
    for seed in range(4096):
        c = orc.quantize(g[0], ex["W"], ex["scales"], seed, idx=idx)
        assert c[0] in (0, 1)
        up += int(c[0])
    p = ex["shared"]["worker0_threshold"] / 2 ** 32
    assert abs(up / 4096 - p) < 6 * math.sqrt(p * (1 - p) / 4096)
    # the deterministic single-worker case |v| = 1/16 at the inclusive tie
    for seed in range(32):
        v = np.array([0.0625], dtype=np.float32)
        k = orc.scale_index_worker(v, ex["W"], ex["scales"])
        assert list(orc.quantize(v, ex["W"], ex["scales"], seed, idx=k)) == [7]


def test_zero_vector_and_non_finite(orc):
    z = np.zeros(37, dtype=np.float32)
    assert not orc.quantize(z, 1.0, [127.0], 5).any()
    v = np.array([np.inf, -np.inf, np.nan, 0.0, -0.0, 0.5], dtype=np.float32)
    c = orc.quantize(v, 1.0, [127.0], 5)
    assert list(c[:5]) == [0] * 5 and c[5] in (63, 64)
    for W in (0.0, np.inf, np.nan, -2.0):
        assert not orc.quantize(v, W, [127.0], 5).any()


@pytest.mark.parametrize("seed", range(3))
def test_codes_in_exact_two_point_support(orc, seed):
    """Every code is sign * floor(x) or sign * (floor(x) + 1) with x = |v| s / W
    in exact arithmetic (up to the binary32 rounding of x at a level edge)."""
    rng = np.random.default_rng(seed)
    W = np.float32(3.0)
    scales = [127.0, 2032.0, 32512.0]
    v = (W * rng.uniform(-1, 1, size=4000) ** 3).astype(np.float32)
    idx = orc.scale_index_worker(v, W, scales)
    c = orc.quantize(v, W, scales, seed=77 + seed, idx=idx)
    Wf = exact.frac(W)
    for vi, ci, ki in zip(v, c, idx):
        xe = abs(exact.frac(vi)) * Fraction(scales[ki]) / Wf
        lo = math.floor(xe)
        allowed = {lo, lo + 1}
        # the binary32 x may cross an integer within its rounding error
        if abs(xe - round(xe)) <= xe * Fraction(1, 2 ** 22):
            allowed |= {round(xe) - 1, round(xe), round(xe) + 1}
        assert abs(int(ci)) in allowed
        assert abs(int(ci)) <= scales[0]
        assert (ci == 0) or (np.sign(ci) == np.sign(vi))


def test_sign_symmetry(orc):
    """The random word depends on (seed, worker, i) only: Q(-v) = -Q(v)."""
    v = np.random.default_rng(2).normal(size=513).astype(np.float32)
    for seed in (0, 1, 2 ** 40 + 5):
        assert np.array_equal(orc.quantize(-v, 4.0, [127.0], seed), -orc.quantize(v, 4.0, [127.0], seed))


def test_window_consistency(orc):
    """Quantising coordinates [i0, i0+n) of a row equals that slice of the whole row."""
    v = np.random.default_rng(9).normal(size=1000).astype(np.float32)
    full = orc.quantize(v, 40.0, [127.0], 3, worker=5)
    for i0, n in ((0, 1), (7, 9), (8, 16), (333, 667), (999, 1)):
        part = orc.quantize(v[i0:i0 + n], 40.0, [127.0], 3, worker=5, i0=i0)
        assert np.array_equal(part, full[i0:i0 + n])


def test_single_scale_equals_one_element_multi(orc):
    v = np.random.default_rng(10).normal(size=777).astype(np.float32)
    a = orc.quantize(v, 30.0, [127.0], 11)
    b = orc.quantize(v, 30.0, [127.0], 11, idx=np.zeros(777, dtype=np.uint8))
    assert np.array_equal(a, b)


@pytest.mark.parametrize("case", ["single", "multi"])
def test_unbiased_over_seeds(orc, case):
    """Lemma 1 / Lemma 2: E[Q(v)] = v.  Mean code over 4096 seeds against
    (i) the exact per-coordinate expectation l + t/2^32 (z-scores) and
    (ii) the paper's expectation a s / W in exact arithmetic."""
    rng = np.random.default_rng(21)
    n = 96
    W = np.float32(2.0)
    v = (W * rng.uniform(-1, 1, size=n) ** 2).astype(np.float32)
    v[:3] = 0.0
    scales = [7.0] if case == "single" else [7.0, 112.0, 1792.0]
    idx = None if case == "single" else orc.scale_index_worker(v, W, scales)
    x, l, t = _x_and_t(v, W, scales, idx)
    seeds = 4096
    total = np.zeros(n)
    for seed in range(seeds):
        total += np.abs(orc.quantize(v, W, scales, seed, idx=idx).astype(np.float64))
    mean = total / seeds
    p = t / 2.0 ** 32
    expect = l + p
    sd = np.sqrt(np.maximum(p * (1 - p), 1e-12) / seeds)
    z = (mean - expect) / sd
    assert np.max(np.abs(z)) < 6
    live = p * (1 - p) > 1e-3
    assert 0.6 < np.mean(z[live] ** 2) < 1.5
    # the realised expectation equals a * s* / W up to binary32 rounding
    k = np.zeros(n, dtype=np.int64) if idx is None else idx
    for i in range(n):
        xe = abs(exact.frac(v[i])) * Fraction(scales[k[i]]) / exact.frac(W)
        ee = Fraction(int(l[i])) + Fraction(int(t[i]), 2 ** 32)
        assert abs(ee - xe) <= xe * Fraction(1, 2 ** 22) + Fraction(1, 2 ** 32)


def test_variance_matches_closed_form_and_lemma_bound(orc):
    rng = np.random.default_rng(31)
    n = 64
    W = np.float32(1.0)
    v = rng.uniform(-1, 1, size=n).astype(np.float32) / np.float32(8)
    s = 7.0
    x, l, t = _x_and_t(v, W, [s])
    p = t / 2.0 ** 32
    closed = float(np.sum((float(W) / s) ** 2 * p * (1 - p)))
    seeds = 3000
    errs = np.zeros(seeds)
    for seed in range(seeds):
        q = float(W) * orc.quantize(v, W, [s], seed).astype(np.float64) / s
        errs[seed] = np.sum((q - v.astype(np.float64)) ** 2)
    se = errs.std() / math.sqrt(seeds)
    assert abs(errs.mean() - closed) < 6 * se
    assert closed <= exact.lemma_bound(n, s, exact.frac(W))
    # the proof's variance (paper's p, exact reals) agrees with the realised one
    proof = float(exact.proof_variance(v, [Fraction(s)] * n, exact.frac(W)))
    assert abs(proof - closed) <= 1e-6 * max(proof, 1e-30)


def test_distinct_workers_and_seeds_decorrelate(orc):
    v = np.full(4096, 0.5, dtype=np.float32)  # p = 1/2 everywhere (s = 3, W = 1)
    a = orc.quantize(v, 1.0, [3.0], 1, worker=0)
    b = orc.quantize(v, 1.0, [3.0], 1, worker=1)
    c = orc.quantize(v, 1.0, [3.0], 2, worker=0)
    for other in (b, c):
        agree = np.mean(a == other)
        assert abs(agree - 0.5) < 6 * 0.5 / math.sqrt(v.size)
