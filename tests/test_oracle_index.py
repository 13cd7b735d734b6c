"""Pins for the oracle's per-coordinate scale rule and scale sharing.

Eq. (11): s*_i is the largest s in S with s <= (W / |v_i|) * min_j s_j.
Scale sharing (Sec. 3.2, Algorithm 2): s*_i = min over workers of s*^m_i.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import exact

HERE = os.path.dirname(os.path.abspath(__file__))
GOLD = json.load(open(os.path.join(HERE, "golden", "worked_examples.json")))


def test_worked_example_D_single_worker(orc):
    ex = GOLD["D"]
    for case in ex["single_worker"]:
        k = orc.scale_index_worker(np.array([case["v"], -case["v"]], dtype=np.float32), ex["W"], ex["scales"])
        assert list(k) == [case["index"], case["index"]]


def test_worked_example_D_sharing(orc):
    ex = GOLD["D"]
    g = np.array(ex["shared"]["rows"], dtype=np.float32)
    idx = orc.scale_index_shared(g, ex["W"], ex["scales"])
    assert list(idx) == [ex["shared"]["index"]]


def test_zero_and_non_finite_take_largest_scale(orc):
    v = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, 0.5], dtype=np.float32)
    k = orc.scale_index_worker(v, 1.0, [7.0, 112.0, 1792.0])
    assert list(k[:5]) == [2] * 5
    assert k[5] == 0  # 0.5 * 112 > 7


def test_zero_path_selects_last_index(orc):
    v = np.array([0.1, 0.2], dtype=np.float32)
    for W in (0.0, np.inf, np.nan):
        assert list(orc.scale_index_worker(v, W, [7.0, 112.0])) == [1, 1]


def test_norm_coordinate_takes_smallest_scale(orc):
    """|v_i| = W: only s_min satisfies s <= s_min, whatever the other scales."""
    v = np.array([2.5, -2.5], dtype=np.float32)
    assert list(orc.scale_index_worker(v, 2.5, [127.0, 2032.0, 32512.0])) == [0, 0]


@pytest.mark.parametrize("seed", range(6))
def test_agrees_with_exact_rule_away_from_ties(orc, seed):
    """The binary32 evaluation of Eq. (11) equals the exact-real rule except
    where |v| s_k / W lies within rounding of s_min."""
    rng = np.random.default_rng(seed)
    scales = [7.0, 112.0, 1792.0, 28672.0] if seed % 2 else [127.0, 2032.0, 32512.0, 520192.0, 127 * 16.0 ** 4]
    W = np.float32(np.exp(rng.uniform(-5, 5)))
    v = (W * np.exp(rng.uniform(-25, 0, size=3000)) * rng.choice([-1, 1], 3000)).astype(np.float32)
    k = orc.scale_index_worker(v, W, scales)
    Wf = exact.frac(W)
    s0 = Fraction(scales[0])
    mismatches = 0
    for vi, ki in zip(v, k):
        a = abs(exact.frac(vi))
        want = exact.exact_scale_index(a, Wf, scales)
        if want != ki:
            # allowed only at a rounding tie of the boundary scale
            kk = max(want, int(ki))
            ratio = a * Fraction(scales[kk]) / Wf / s0
            assert abs(ratio - 1) < Fraction(1, 2 ** 21), (vi, want, ki)
            mismatches += 1
    assert mismatches <= 3


@pytest.mark.parametrize("seed", range(4))
def test_sharing_invariants(orc, seed):
    rng = np.random.default_rng(100 + seed)
    M, d = 5, 2000
    scales = [127.0, 2032.0, 32512.0, 520192.0]
    g = (rng.normal(size=(M, d)) * 10.0 ** rng.uniform(-6, 0, size=(M, d))).astype(np.float32)
    g[rng.random((M, d)) < 0.05] = 0.0
    W, _ = orc.shared_scale(g)
    idx = orc.scale_index_shared(g, W, scales)
    own = np.stack([orc.scale_index_worker(g[m], W, scales) for m in range(M)])
    assert np.array_equal(idx, own.min(axis=0))
    assert idx.max() <= len(scales) - 1
    inv = (np.array(scales, dtype=np.float32) / W).astype(np.float32)
    amax = np.abs(g).max(axis=0)
    s0 = np.float32(scales[0])
    for i in range(d):
        k = idx[i]
        if amax[i] == 0:
            assert k == len(scales) - 1
            continue
        # feasibility for every worker (x <= s_min) and maximality for the limiting worker
        assert np.all(np.abs(g[:, i]) * inv[k] <= s0) or k == 0
        if k + 1 < len(scales):
            assert np.float32(amax[i] * inv[k + 1]) > s0


def test_single_scale_has_index_zero(orc):
    v = np.random.default_rng(1).normal(size=100).astype(np.float32)
    assert not orc.scale_index_worker(v, 20.0, [127.0]).any()
