"""Exact-arithmetic helpers for the oracle's pins (test code only).

These compute the paper's definitions with Python ``Fraction`` (no rounding) or
by brute force, so that a mistake in the oracle's floating-point realisation
shows up as a disagreement instead of being copied.
"""
from __future__ import annotations

import itertools
import math
import struct
from fractions import Fraction

import numpy as np


def f32(x) -> float:
    return struct.unpack("<f", struct.pack("<f", float(x)))[0]


def round_half_even(x: Fraction) -> int:
    fl = math.floor(x)
    d = x - fl
    if d > Fraction(1, 2):
        return fl + 1
    if d < Fraction(1, 2):
        return fl
    return fl if fl % 2 == 0 else fl + 1


def fp32_from_fraction(x: Fraction) -> float:
    """Exact round-to-nearest-even of a rational to fp32 (normal and subnormal)."""
    if x == 0:
        return 0.0
    sign = -1.0 if x < 0 else 1.0
    a = abs(x)
    e = math.floor(math.log2(a.numerator) - math.log2(a.denominator))
    # fix e so that 2^e <= a < 2^(e+1)
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    e = max(e, -126)
    step = Fraction(2) ** (e - 23)
    n = round_half_even(a / step)
    return sign * float(n * step)


def rtn_codes_exact(w, lo: Fraction, s: Fraction, qmax: int):
    """Eq. rtn with exact arithmetic: clamp(round((w - lo)/s), 0, qmax).
    Also returns each element's distance from the nearest rounding boundary
    (in code units), so callers can excuse boundary cases."""
    codes, dist = [], []
    for wi in w:
        x = (Fraction(float(wi)) - lo) / s
        q = min(max(round_half_even(x), 0), qmax)
        codes.append(q)
        # only the boundaries k + 1/2 with 0 <= k < qmax change a clamped code
        if x <= Fraction(-1, 2) or x >= qmax + Fraction(1, 2):
            dist.append(math.inf)
        else:
            frac = x - math.floor(x)
            dist.append(float(abs(frac - Fraction(1, 2))))
    return np.array(codes), np.array(dist)


def wls_fit(q, w, h):
    """Weighted least squares r = s q + z via numpy's lstsq on sqrt(h)-scaled
    rows (a library routine independent of the oracle's closed form)."""
    q = np.asarray(q, np.float64)
    w = np.asarray(w, np.float64)
    sh = np.sqrt(np.asarray(h, np.float64))
    A = np.stack([q * sh, sh], axis=1)
    sol, *_ = np.linalg.lstsq(A, w * sh, rcond=None)
    return float(sol[0]), float(sol[1])


def score(q, w, h, s, z):
    q = np.asarray(q, np.float64)
    w = np.asarray(w, np.float64)
    h = np.asarray(h, np.float64)
    e = s * q + z - w
    return float(np.sum(h * e * e))


def monotone_assignments(n: int, qmax: int):
    """Every non-decreasing code sequence of length n over 0..qmax."""
    for comb in itertools.combinations_with_replacement(range(qmax + 1), n):
        yield np.array(comb)


E2M1_LEVELS = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])


def e2m1_nearest_index(a: float) -> int:
    """Brute-force nearest E2M1 magnitude index for |y| = a, ties to the even
    index (the level whose mantissa bit is 0), saturating at 6."""
    a = Fraction(float(a))
    d = [abs(Fraction(float(l)) - a) for l in E2M1_LEVELS]
    dmin = min(d)
    best = [i for i, x in enumerate(d) if x == dmin]
    if len(best) == 1:
        return best[0]
    return [b for b in best if b % 2 == 0][0]


def e4m3_levels():
    """All non-negative finite E4M3FN values with their bytes (brute force)."""
    vals = []
    for code in range(0x7F):  # 0x7F is NaN
        e, m = (code >> 3) & 15, code & 7
        v = m * 2.0 ** -9 if e == 0 else (1 + m / 8) * 2.0 ** (e - 7)
        vals.append((v, code))
    return vals


def sqrt_fp32(x: float) -> float:
    """Correctly rounded fp32 square root of the fp32 value x >= 0 (nearest,
    ties to even), decided with exact rational comparisons of the midpoints."""
    x = float(np.float32(x))
    if x == 0.0:
        return 0.0
    c = np.float32(math.sqrt(x))
    cands = [np.nextafter(c, np.float32(0)), c, np.nextafter(c, np.float32(np.inf))]
    fx = Fraction(x)
    best = None
    for r in cands:
        lo = (Fraction(float(np.nextafter(r, np.float32(0)))) + Fraction(float(r))) / 2
        hi = (Fraction(float(r)) + Fraction(float(np.nextafter(r, np.float32(np.inf))))) / 2
        if lo * lo < fx < hi * hi:
            return float(r)
        if fx == lo * lo or fx == hi * hi:  # a tie: the even neighbour
            if int(np.float32(r).view(np.uint32)) % 2 == 0:
                best = float(r)
    assert best is not None
    return best
