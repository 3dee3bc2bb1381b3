"""Rank sets that stress the single rounding of the mean gradient, and its
exact value from Python's rational arithmetic.

The mean gradient is g_bar = fp32(S / R) with S the exact sum of R BF16
values, rounded once (round to nearest, ties to even).  Three kinds of rank
sets make that rounding hard:
  - near_midpoint: S / R lies on an FP32 midpoint, or a tiny value away from
    one, with cancelling pairs of large values mixed in, in random rank order,
    so that an FP64 sum in rank order is often inexact;
  - wide_span: random finite BF16 values over the whole exponent range;
  - subnormal_remainder: S / R in the FP32 subnormal range where the integer
    part of the quotient sits exactly on a midpoint and only the remainder of
    the division by R says which way to round.
Nothing here computes the mean the way the oracle or the library does; the
expected value comes from fractions.Fraction.
"""
from fractions import Fraction

import numpy as np


def bf16_fraction(b: int) -> Fraction:
    """Exact value of a finite BF16 bit pattern."""
    b = int(b)
    sign = -1 if b & 0x8000 else 1
    e, f = (b >> 7) & 0xFF, b & 0x7F
    assert e != 0xFF, "not finite"
    if e == 0:
        return sign * Fraction(f, 1 << 133)
    return sign * Fraction(0x80 | f) * Fraction(2) ** (e - 134)


def bf16_of_fraction(x: Fraction) -> int:
    """BF16 pattern of a value that BF16 represents exactly (asserted)."""
    if x == 0:
        return 0
    sign = 0x8000 if x < 0 else 0
    a = abs(x)
    # normalise a = M * 2^k with 128 <= M < 256, or a subnormal
    k = a.numerator.bit_length() - a.denominator.bit_length() - 8
    while Fraction(2) ** (k + 8) <= a:
        k += 1
    while Fraction(2) ** (k + 7) > a:
        k -= 1
    if k < -133:
        k = -133
    M = a / Fraction(2) ** k
    assert M.denominator == 1 and M < 256, "not representable in BF16"
    M = int(M)
    if M < 128:
        assert k == -133
        return sign | M
    e = k + 134
    assert 1 <= e <= 254
    return sign | (e << 7) | (M & 0x7F)


def rne32(x: Fraction) -> np.float32:
    """Round a rational to the nearest FP32 value, ties to the even pattern."""
    if x == 0:
        return np.float32(0.0)
    a = np.float32(float(x))  # within one FP32 step of the answer
    cands = {a, np.nextafter(a, np.float32(-np.inf)), np.nextafter(a, np.float32(np.inf))}
    best = None
    for c in cands:
        if not np.isfinite(c):
            continue
        d = abs(Fraction(float(c)) - x)
        key = (d, int(np.array(c, np.float32).view(np.uint32)) & 1)
        if best is None or key < best[0]:
            best = (key, c)
    return np.float32(best[1])


def exact_mean(bits_col) -> np.float32:
    """fp32(S / R) of one element's R BF16 patterns; +0 for S = 0."""
    s = sum(bf16_fraction(b) for b in bits_col)
    return rne32(s / len(bits_col))


def exact_means(ranks: np.ndarray) -> np.ndarray:
    """ranks: (R, n) uint16 -> (n,) float32 of the exact rounded means."""
    return np.array([exact_mean(ranks[:, i]) for i in range(ranks.shape[1])], np.float32)


def rank_order_f64_mean(ranks: np.ndarray) -> np.ndarray:
    """The double-rounded candidate: FP64 sum in rank order, FP64 divide, then FP32."""
    vals = (ranks.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    s = np.zeros(ranks.shape[1])
    for r in range(ranks.shape[0]):
        s = s + vals[r]
    return (s / ranks.shape[0]).astype(np.float32)


def _random_bf16(rng, lo_e=1, hi_e=254):
    e = int(rng.integers(lo_e, hi_e + 1))
    return (int(rng.integers(0, 2)) << 15) | (e << 7) | int(rng.integers(0, 128))


def near_midpoint(R: int, n: int, seed: int) -> np.ndarray:
    """n rank sets whose mean is an FP32 midpoint 2^E + (2k+1) 2^(E-24), or
    that plus or minus one tiny value, written as R BF16 values: R 2^E,
    R (2k+1) 2^(E-24), the tiny value, and cancelling pairs +x, -x; shuffled."""
    assert R >= 3
    rng = np.random.default_rng(seed)
    out = np.zeros((R, n), np.uint16)
    for i in range(n):
        E = int(rng.integers(-100, 100))
        k = int(rng.integers(0, (255 // R - 1) // 2 + 1))
        sgn = -1 if rng.integers(0, 2) else 1
        A = sgn * R * Fraction(2) ** E
        B = sgn * R * (2 * k + 1) * Fraction(2) ** (E - 24)
        d = int(rng.choice([0, 0, 20, 30, 45, 50, 52, 53, 54, 55, 60, 80, 110]))
        if d == 0 or E - d < -133:
            delta = Fraction(0)
        else:
            delta = (1 if rng.integers(0, 2) else -1) * Fraction(2) ** (E - d)
        vals = [A, B, delta]
        while len(vals) < R:
            if len(vals) + 2 <= R:
                x = bf16_fraction(_random_bf16(rng, 1, 254) & 0x7FFF)
                vals += [x, -x]
            else:
                vals.append(Fraction(0))
        order = rng.permutation(R)
        for r in range(R):
            out[r, i] = bf16_of_fraction(vals[order[r]])
    return out


def wide_span(R: int, n: int, seed: int) -> np.ndarray:
    """n rank sets of independent random finite BF16 values, every exponent."""
    rng = np.random.default_rng(seed)
    out = np.zeros((R, n), np.uint16)
    for i in range(n):
        for r in range(R):
            out[r, i] = _random_bf16(rng, 0, 254)
    return out


def subnormal_remainder(R: int, limit: int = 4000) -> np.ndarray:
    """Rank sets of subnormal values whose sum S = K 2^-133 gives a quotient
    S / R below 2^-126 whose bits down to 2^-153 end exactly on a midpoint of
    the 2^-149 grid while S / R is not a multiple of 2^-153: only the division's
    remainder decides the rounding.  Also the neighbouring K - 1 and K + 1."""
    ks = []
    for K in range(1, limit):
        units = K << 20                # S in units of 2^-153
        Q, rem = divmod(units, R)
        if rem != 0 and (Q & 0xF) == 0x8:
            ks += [K - 1, K, K + 1]
    cols = []
    for K in ks:
        if K < 1 or K > 127 * R:
            continue
        col, left = [], K
        for r in range(R):
            take = min(127, left - 0)
            col.append(take)
            left -= take
        if left == 0:
            cols.append(col)
    out = np.array(cols, dtype=np.uint16).T.copy() if cols else np.zeros((R, 0), np.uint16)
    return out


def remainder_decides(ranks: np.ndarray) -> int:
    """How many of subnormal_remainder's sets round up only because of the
    remainder: their truncated quotient's tie would go down to even."""
    n = 0
    R = ranks.shape[0]
    for i in range(ranks.shape[1]):
        K = sum(int(x) for x in ranks[:, i])
        Q, rem = divmod(K << 20, R)
        n += bool(rem and (Q & 0xF) == 0x8 and ((Q >> 4) & 1) == 0)
    return n
