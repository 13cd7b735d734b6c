"""Pins for the oracle's integer all-reduce and reconstruction.

Algorithm 1/2: zeta_t = (1/M) sum_m zeta^m (an exact integer sum of the codes
with the 1/M folded into the reconstruction), ghat = R(zeta) = W * zeta / s*
(Eq. (9) and Eq. (13)).  The scheme commutes with aggregation (Sec. 3.1):
reconstructing the summed codes equals averaging per-worker reconstructions.
Brute force over all 2^n outcomes pins E[Q(v)] = v and the variance bound
of Lemma 1 / Lemma 2 exactly.
"""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import exact
from tests.conftest import ulp_distance_f32

HERE = os.path.dirname(os.path.abspath(__file__))
GOLD = json.load(open(os.path.join(HERE, "golden", "worked_examples.json")))


def test_sum_is_integer_identity(orc):
    rng = np.random.default_rng(1)
    codes = rng.integers(-127, 128, size=(9, 1000)).astype(np.int8)
    assert np.array_equal(orc.sum_codes(codes), codes.astype(np.int64).sum(axis=0))
    # a strided view (leading dimension > d) sums only the first d coordinates
    assert np.array_equal(orc.sum_codes(codes, d=513), codes[:, :513].astype(np.int64).sum(axis=0))


def test_sum_brute_force_tiny():
    """Every int8 triple at a handful of coordinates, summed by enumeration."""
    from oracle import oracle as O

    vals = [-128, -127, -1, 0, 1, 126, 127]
    for combo in itertools.product(vals, repeat=3):
        codes = np.array(combo, dtype=np.int8).reshape(3, 1)
        assert O.sum_codes(codes)[0] == sum(combo)


def test_example_A_reconstruction(orc):
    ex = GOLD["A"]
    g = np.array(ex["rows"], dtype=np.float32)
    r = orc.pipeline(g, ex["scales"], seed=123)
    assert list(r["sum"]) == ex["sum"]
    assert list(r["out"]) == ex["out"]
    zero, inv, deq = orc.tables(r["W"], ex["scales"], M=1)
    assert deq[0] == np.float32(ex["deq"])
    g2 = np.concatenate([g, g])
    r2 = orc.pipeline(g2, ex["scales"], seed=123)
    assert list(r2["sum"]) == ex["two_identical_rows"]["sum"]
    assert list(r2["out"]) == ex["two_identical_rows"]["out"]
    assert orc.tables(r2["W"], ex["scales"], M=2)[2][0] == np.float32(ex["two_identical_rows"]["deq"])


@pytest.mark.parametrize("scales", [[127.0], [7.0, 112.0, 1792.0, 28672.0]])
def test_commutes_with_aggregation(orc, scales):
    """dequant(sum_m codes) vs mean_m dequant(codes^m): equal up to a few ulp
    (Sec. 3.1: the compression commutes with gradient aggregation)."""
    rng = np.random.default_rng(5)
    M, d = 6, 3000
    g = (rng.normal(size=(M, d)) * 1e-3).astype(np.float32)
    r = orc.pipeline(g, scales, seed=9)
    per_worker = np.stack([orc.dequantize(r["codes"][m].astype(np.int32), 1, r["W"], scales, r["idx"])
                           for m in range(M)]).astype(np.float64)
    mean = per_worker.mean(axis=0)
    diff = np.abs(r["out"].astype(np.float64) - mean)
    # each side carries two binary32 roundings of terms no larger than the
    # workers' own reconstructions; cancellation in the sum does not shrink them
    scale = np.abs(r["out"]).astype(np.float64) + np.abs(per_worker).mean(axis=0)
    assert np.all(diff <= scale * 2.0 ** -21)


def test_dequantize_exact_value(orc):
    """out_i = RN32(sum_i * RN32(W / (M s*_i))) checked in exact arithmetic."""
    rng = np.random.default_rng(8)
    scales = [127.0, 2032.0, 32512.0]
    W = np.float32(0.37)
    sums = rng.integers(-8 * 127, 8 * 127 + 1, size=500).astype(np.int32)
    idx = rng.integers(0, 3, size=500).astype(np.uint8)
    out = orc.dequantize(sums, 8, W, scales, idx)
    for s_i, k, o in zip(sums, idx, out):
        dq = exact.round_f32(exact.frac(W) / (8 * Fraction(scales[k])))
        q = Fraction(int(s_i)) * exact.frac(dq)
        want = exact.round_f32(abs(q))
        assert abs(o) == want and (o == 0 or np.sign(o) == np.sign(s_i))
    # the reconstruction itself is within two roundings of W * sum / (M s*)
    for s_i, k, o in zip(sums, idx, out):
        real = exact.frac(W) * int(s_i) / (8 * Fraction(scales[k]))
        assert abs(exact.frac(o) - real) <= abs(real) * Fraction(1, 2 ** 22)


def test_averaged_gradient_is_unbiased(orc):
    """E[ghat] = (1/M) sum_m g^m (Sec. 3.1 averaging with Lemma 1)."""
    rng = np.random.default_rng(12)
    M, d = 4, 256
    g = (rng.normal(size=(M, d)) * 1e-2).astype(np.float32)
    target = g.astype(np.float64).mean(axis=0)
    W, _ = orc.shared_scale(g)
    s = 7.0
    seeds = 2000
    acc = np.zeros(d)
    for seed in range(seeds):
        acc += orc.pipeline(g, [s], seed=seed)["out"]
    mean = acc / seeds
    # per-coordinate sd of ghat <= W / (M s) * sqrt(M) / 2 per draw
    sd = float(W) / (M * s) * math.sqrt(M) * 0.5 / math.sqrt(seeds)
    assert np.max(np.abs(mean - target)) < 6 * sd


def test_zero_inputs_reconstruct_to_zero(orc):
    r = orc.pipeline(np.zeros((3, 50), dtype=np.float32), [127.0, 2032.0], seed=1)
    assert r["W"] == 0 and not r["codes"].any() and not r["out"].any()
    assert np.all(r["idx"] == 1)


# --------------------------------------------------------------------------
# Brute force over all 2^n outcomes (exact rationals)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("seed", list(range(8)) + [8, 9])
def test_brute_force_moments_and_lemma(orc, seed):
    rng = np.random.default_rng(1000 + seed)
    # seeds 8 and 9: d = 16, all 65536 outcomes
    n = int(rng.integers(3, 11)) if seed < 8 else 16
    multi = seed % 2 == 1
    scales = [3.0, 48.0] if multi else [float(rng.integers(1, 9))]
    v = (rng.normal(size=n) * 0.3).astype(np.float32)
    v[0] = 0.0
    W = exact.exact_max_norm(v.reshape(1, -1))
    W_orc, _ = orc.shared_scale(v.reshape(1, -1))
    assert ulp_distance_f32(W_orc, W) <= 1
    W = W_orc
    idx = orc.scale_index_worker(v, W, scales) if multi else None
    x, l, t = _xt(v, W, scales, idx)
    s_star = [Fraction(scales[0 if idx is None else idx[i]]) for i in range(n)]
    laws = [(int(l[i]), Fraction(int(t[i]), 2 ** 32)) for i in range(n)]
    Wf = exact.frac(W)
    mean, second = exact.brute_force_moments(v, s_star, Wf, laws)
    # unbiasedness up to the binary32 rounding of x = |v| s / W
    for i in range(n):
        vi = exact.frac(v[i])
        assert abs(mean[i] - vi) <= abs(vi) * Fraction(1, 2 ** 21) + Wf / s_star[i] / 2 ** 32
    # exact second moment = the proof's closed form with the realised p, plus
    # the squared rounding bias of each coordinate's mean
    closed = sum((Wf / s_star[i]) ** 2 * laws[i][1] * (1 - laws[i][1]) for i in range(n))
    bias2 = sum((mean[i] - exact.frac(v[i])) ** 2 for i in range(n))
    assert second == closed + bias2
    assert float(second) <= exact.lemma_bound(n, min(scales), Wf)
    # every oracle draw lies in the support of the enumerated law
    for sd in range(64):
        c = orc.quantize(v, W, scales, sd, idx=idx)
        for i in range(n):
            assert abs(int(c[i])) in (laws[i][0], laws[i][0] + 1)


def _xt(v, W, scales, idx):
    s = np.asarray(scales, dtype=np.float32)
    k = np.zeros(v.size, dtype=np.int64) if idx is None else idx.astype(np.int64)
    inv = (s / np.float32(W)).astype(np.float32)
    x = np.minimum(np.abs(v) * inv[k], s[0]).astype(np.float32)
    l = np.floor(x)
    t = ((x - l).astype(np.float64) * 2.0 ** 32).astype(np.uint64)
    return x, l.astype(np.int64), t
