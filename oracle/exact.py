"""TEST INFRASTRUCTURE ONLY: exact rational arithmetic for pinning the oracle.

Everything here is computed with Python integers and fractions.Fraction, so
it carries no floating-point rounding except where a result is explicitly
rounded to binary32 (round-to-nearest, ties-to-even) by `round_f32`.  It is
independent of the C oracle and is used only by the tests.

Sources: the quantiser Q_s of Eq. (7)-(8) (Sec. 3.1), the scale rule Eq. (11)
and sharing rule (Sec. 3.2), the reconstruction Eq. (9)/(13), and the
unbiasedness/variance statements of Lemma 1 and Lemma 2 with their proofs
(Appendix C and E).
"""
from __future__ import annotations

import itertools
import math
from fractions import Fraction

import numpy as np

F32_MAX = Fraction(2) ** 127 * (2 - Fraction(1, 2 ** 23))


def frac(x) -> Fraction:
    """The exact value of a binary32/binary64 number."""
    return Fraction(float(x))


def _f32_neighbours(x: np.float32):
    lo = np.nextafter(x, np.float32(-np.inf), dtype=np.float32)
    hi = np.nextafter(x, np.float32(np.inf), dtype=np.float32)
    return lo, hi


def round_f32(q: Fraction) -> np.float32:
    """Correctly rounded binary32 value of a non-negative rational q (finite range)."""
    assert q >= 0
    if q == 0:
        return np.float32(0.0)
    if q > F32_MAX:
        # overflow threshold: F32_MAX + half an ulp rounds to infinity
        if q >= F32_MAX + Fraction(2) ** 103:
            return np.float32(np.inf)
        return np.float32(F32_MAX)
    # start from a nearby binary32 and walk until q lies within half an ulp
    c = np.float32(float(q))
    for _ in range(8):
        lo, hi = _f32_neighbours(c)
        below = (frac(lo) + frac(c)) / 2
        above = (frac(c) + frac(hi)) / 2
        if q < below:
            c = lo
        elif q > above:
            c = hi
        elif q == below or q == above:
            # tie: choose the neighbour with an even significand
            other = lo if q == below else hi
            c_bits = int(np.array(c, dtype=np.float32).view(np.uint32))
            return c if c_bits % 2 == 0 else other
        else:
            return c
    raise AssertionError("round_f32 did not converge")


def sqrt_round_f32(S: Fraction) -> np.float32:
    """Correctly rounded binary32 value of sqrt(S) for a rational S >= 0."""
    assert S >= 0
    if S == 0:
        return np.float32(0.0)
    c = np.float32(math.sqrt(float(S)))
    for _ in range(8):
        lo, hi = _f32_neighbours(c)
        below = ((frac(lo) + frac(c)) / 2) ** 2
        above = ((frac(c) + frac(hi)) / 2) ** 2
        if S < below:
            c = lo
        elif S > above:
            c = hi
        else:
            # a rational square root equal to a binary32 midpoint would need
            # S to be the square of a 25-bit dyadic: handle it as a tie
            if S == below or S == above:
                other = lo if S == below else hi
                c_bits = int(np.array(c, dtype=np.float32).view(np.uint32))
                return c if c_bits % 2 == 0 else other
            return c
    raise AssertionError("sqrt_round_f32 did not converge")


def exact_sum_of_squares(v) -> Fraction:
    return sum((frac(x) ** 2 for x in np.asarray(v, dtype=np.float32).reshape(-1)), Fraction(0))


def exact_max_norm(g) -> np.float32:
    """RN_f32( max_m ||g^m||_2 ) computed exactly (Sec. 3.1: ||w|| = max_m ||g^m||)."""
    g = np.asarray(g, dtype=np.float32)
    return sqrt_round_f32(max(exact_sum_of_squares(row) for row in g))


def exact_scale_index(a: Fraction, W: Fraction, scales) -> int:
    """Eq. (11) in exact arithmetic: the largest k with s_k <= (W/a) * s_min.

    a == 0 selects the largest scale (every scale satisfies the rule).  No
    qualifying scale (only possible if a > W) selects index 0.
    """
    s = [frac(x) for x in scales]
    if a == 0:
        return len(s) - 1
    best = 0
    for k, sk in enumerate(s):
        if sk * a <= W * s[0]:
            best = k
    return best


def level_and_prob(x: Fraction):
    """Eq. (8): x = a*s in [l, l+1) -> (l, p = x - l); x == s_max edge uses l = x, p = 0."""
    l = math.floor(x)
    return l, x - l


def outcome_distribution(x_values, t_values=None):
    """Independent per-coordinate two-point laws.

    With t_values None: P(up) = x - floor(x) exactly (the paper's p).
    With t_values given: P(up) = t / 2^32 (what a 32-bit uniform word r with
    the rule r < t realises).  Returns a list of (l_i, P(up)_i).
    """
    laws = []
    for j, x in enumerate(x_values):
        l, p = level_and_prob(x)
        if t_values is not None:
            p = Fraction(int(t_values[j]), 2 ** 32)
        laws.append((l, p))
    return laws


def enumerate_outcomes(laws):
    """Brute force over all 2^n joint outcomes of independent two-point laws.

    Yields (magnitudes tuple, probability) for every joint outcome.
    """
    for ups in itertools.product((0, 1), repeat=len(laws)):
        prob = Fraction(1)
        mags = []
        for (l, p), u in zip(laws, ups):
            prob *= p if u else (1 - p)
            mags.append(l + u)
        yield tuple(mags), prob


def brute_force_moments(v, scale_per_coord, W: Fraction, laws):
    """Exact E[Q(v)] and E||Q(v) - v||^2 over all 2^n outcomes.

    Q_i = W * sign(v_i) * mag_i / s*_i  (Eq. (7)/(10) with xi = mag / s*).
    Every joint outcome is enumerated; its probability is carried as an
    integer numerator over 2^(32 n) (each p_i is a multiple of 2^-32), and
    each coordinate accumulates the probability mass of its upper level.
    """
    v = [frac(x) for x in v]
    n = len(v)
    one = 1 << 32
    weights = []
    for _, p in laws:
        a = p * one
        assert a.denominator == 1 and 0 <= a <= one
        weights.append((one - int(a), int(a)))
    total = 0
    upper = [0] * n  # sum of the probabilities of the outcomes with mag_i = l_i + 1
    for ups in itertools.product((0, 1), repeat=n):
        prob = 1
        for (w0, w1), u in zip(weights, ups):
            prob *= w1 if u else w0
        total += prob
        for i, u in enumerate(ups):
            if u:
                upper[i] += prob
    denom = one ** n
    assert total == denom
    mean = []
    second = Fraction(0)
    for i, (l, _) in enumerate(laws):
        sgn = (v[i] > 0) - (v[i] < 0)
        q0 = W * sgn * Fraction(l) / scale_per_coord[i]
        q1 = W * sgn * Fraction(l + 1) / scale_per_coord[i]
        m0, m1 = Fraction(denom - upper[i], denom), Fraction(upper[i], denom)
        mean.append(m0 * q0 + m1 * q1)
        second += m0 * (q0 - v[i]) ** 2 + m1 * (q1 - v[i]) ** 2
    return mean, second


def lemma_bound(n: int, s_hat, W: Fraction) -> float:
    """(1 + min(n / s^2, sqrt(n) / s)) * ||w||^2 of Lemma 1 / Lemma 2."""
    s_hat = float(s_hat)
    return (1.0 + min(n / s_hat ** 2, math.sqrt(n) / s_hat)) * float(W) ** 2


def proof_variance(v, scale_per_coord, W: Fraction) -> Fraction:
    """The exact variance the proof of Lemma 1 derives: sum_i (W/s*_i)^2 p_i (1 - p_i)."""
    total = Fraction(0)
    for x, s in zip(v, scale_per_coord):
        a = abs(frac(x))
        if a == 0:
            continue
        l, p = level_and_prob(a * s / W)
        total += (W / s) ** 2 * p * (1 - p)
    return total
