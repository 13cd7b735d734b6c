"""Pins for the oracle's shared scale and derived tables.

Shared scale: ||w||_2 = max_m ||g^m||_2 (Sec. 3.1 and 3.2; the MaxAllReduce of
Algorithm 1 and Algorithm 2).  Tables: inv_k = s_k / W (the factor in
a * s = |v| s / W of Eq. (8)) and deq_k = W / (M s_k) (Eq. (9)/(13) with the
1/M of the averaging all-reduce).
"""
from fractions import Fraction

import numpy as np
import pytest

from oracle import exact
from tests.conftest import ulp_distance_f32


def test_closed_form_pythagorean_row(orc):
    g = np.array([[3, -4, 0, 0]], dtype=np.float32) * np.float32(2.0 ** -10)
    W, S = orc.shared_scale(g)
    assert W == np.float32(5 * 2.0 ** -10)
    assert S[0] == 25 * 2.0 ** -20


def test_max_not_sum_over_workers(orc):
    g = np.zeros((3, 8), dtype=np.float32)
    g[0, 0] = 3.0
    g[1, 1] = 12.0
    g[1, 2] = 5.0  # row norm 13
    g[2, :] = 1.0  # row norm sqrt(8)
    W, _ = orc.shared_scale(g)
    assert W == np.float32(13.0)


def test_zero_and_empty(orc):
    W, _ = orc.shared_scale(np.zeros((4, 16), dtype=np.float32))
    assert W == 0.0
    W, _ = orc.shared_scale(np.zeros((2, 16), dtype=np.float32), d=0)
    assert W == 0.0


def test_non_finite_rows_propagate(orc):
    g = np.ones((2, 4), dtype=np.float32)
    g[1, 2] = np.inf
    assert np.isinf(orc.shared_scale(g)[0])
    g[0, 1] = np.nan
    assert np.isnan(orc.shared_scale(g)[0])


@pytest.mark.parametrize("seed", range(40))
def test_brute_force_exact_norm_within_one_ulp(orc, seed):
    """Exact rational sum of squares and exactly rounded sqrt vs the oracle."""
    rng = np.random.default_rng(seed)
    M, d = int(rng.integers(1, 5)), int(rng.integers(1, 17))
    mant = rng.normal(size=(M, d))
    expo = rng.integers(-30, 30, size=(M, d)).astype(np.float64)
    g = (mant * 2.0 ** expo).astype(np.float32)
    W, S = orc.shared_scale(g)
    for m in range(M):
        assert Fraction(S[m]) == exact.exact_sum_of_squares(g[m]) or abs(
            Fraction(S[m]) - exact.exact_sum_of_squares(g[m])) <= Fraction(S[m]) * Fraction(d, 2 ** 52)
    want = exact.exact_max_norm(g)
    assert ulp_distance_f32(W, want) <= 1


def test_brute_force_mostly_exactly_rounded(orc):
    """On short rows the fp64 sum is almost always exact: W is the correctly
    rounded norm in nearly every case (a looser reading of the rounding would
    break this)."""
    rng = np.random.default_rng(7)
    hits = 0
    trials = 300
    for _ in range(trials):
        g = rng.normal(size=(2, 6)).astype(np.float32)
        W, _ = orc.shared_scale(g)
        hits += W == exact.exact_max_norm(g)
    assert hits >= trials - 3


def test_large_row_against_numpy_float64(orc):
    rng = np.random.default_rng(11)
    g = (rng.standard_t(3, size=(3, 1 << 20)) * 1e-4).astype(np.float32)
    W, S = orc.shared_scale(g)
    ref = np.float32(np.sqrt(np.max(np.sum(g.astype(np.float64) ** 2, axis=1))))
    assert ulp_distance_f32(W, ref) <= 1
    for m in range(3):
        assert W >= np.float32(np.sqrt(np.sum(g[m].astype(np.float64) ** 2))) * np.float32(1 - 2 ** -23)


def test_leading_dimension_padding_is_ignored(orc):
    rng = np.random.default_rng(5)
    g = np.full((3, 40), 1e6, dtype=np.float32)
    g[:, :33] = rng.normal(size=(3, 33)).astype(np.float32)
    W_pad, _ = orc.shared_scale(g, d=33)
    W_cut, _ = orc.shared_scale(np.ascontiguousarray(g[:, :33]))
    assert W_pad == W_cut


# --------------------------------------------------------------------------
# Tables
# --------------------------------------------------------------------------

def test_inverse_table_is_correctly_rounded_division(orc):
    rng = np.random.default_rng(3)
    scales = np.array([7.0, 112.0, 1792.0, 28672.0, 127 * 16.0 ** 7], dtype=np.float32)
    for _ in range(2000):
        W = np.float32(np.exp(rng.uniform(-60, 60)))
        zero, inv, deq = orc.tables(W, scales, M=3)
        assert not zero
        assert np.array_equal(inv, scales / W)  # numpy binary32 division is IEEE


def test_dequant_table_is_exactly_rounded_quotient(orc):
    rng = np.random.default_rng(4)
    scales = [127.0, 2032.0, 32512.0, 520192.0]
    for _ in range(500):
        W = np.float32(np.exp(rng.uniform(-30, 30)))
        M = int(rng.integers(1, 64))
        zero, inv, deq = orc.tables(W, scales, M=M)
        for k, s in enumerate(scales):
            want = exact.round_f32(exact.frac(W) / (M * Fraction(s)))
            assert deq[k] == want, (W, M, s)


@pytest.mark.parametrize("W", [0.0, -1.0, np.inf, np.nan, 1e-45])
def test_zero_path_tables(orc, W):
    """W not positive-finite, or s_min / W overflowing, selects the zero path."""
    zero, inv, deq = orc.tables(np.float32(W), [127.0, 2032.0], M=2)
    assert zero
    assert not inv.any() and not deq.any()
