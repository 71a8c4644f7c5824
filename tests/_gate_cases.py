"""Gate inputs whose logits sit at float32 rounding midpoints, and the test
for an exact float64 dot product (test infrastructure; no method
arithmetic).

The gate logit is the float32 value nearest the exact dot product of a bf16
token row and a bf16 gate row (§2.1; rounding reading R3). Both the kernel
and the oracle sum the products in float64 and round once. A bf16 x bf16
product has at most 16 significant bits, so every product is an integer
multiple of 2^e, e the lowest set bit over all products; when the sum of
|products| stays below 2^(53 + e), every partial sum, in any order and any
association, is such a multiple below 2^53 * 2^e and is therefore exact in
float64. Then both sides round the exact value and agree by construction.

``engineered`` builds rows whose exact dot products lie just above, exactly
on, or just below a float32 midpoint (2^-40 away), with large terms that
cancel (a float32 accumulator loses the small ones), and returns the
correctly rounded float32 logits computed with exact rational arithmetic.
"""
from fractions import Fraction

import numpy as np

W_ONE = 0x3F80  # bf16 1.0


def f32_to_bf16_bits(a) -> np.ndarray:
    """float32 -> bf16 bit patterns, round to nearest even (finite inputs)."""
    u = np.asarray(a, np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def _bits_to_f64(bits) -> np.ndarray:
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def bf16_value(bits: int) -> Fraction:
    return Fraction(float(np.array([int(bits) << 16], np.uint32).view(np.float32)[0]))


def bf16_from_dyadic(n: int, e: int) -> int:
    """bf16 bits of n * 2^e for |n| <= 256 (exactly representable)."""
    assert abs(n) <= 256
    v = np.float32(n) * np.float32(2.0) ** e
    assert Fraction(float(v)) == Fraction(n) * Fraction(2) ** e
    b = int(np.array([v], np.float32).view(np.uint32)[0])
    assert b & 0xFFFF == 0
    return b >> 16


def round_f32(v: Fraction) -> Fraction:
    """Nearest float32 to an exact rational (normal range), ties to even."""
    if v == 0:
        return Fraction(0)
    s = -1 if v < 0 else 1
    a = abs(v)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1
    ulp = Fraction(2) ** (e - 23)
    q, r = divmod(a, ulp)
    q = int(q)
    if r * 2 > ulp or (r * 2 == ulp and q % 2 == 1):
        q += 1
    return s * q * ulp


def lsb_exponents(bits: np.ndarray) -> np.ndarray:
    """Exponent of the lowest set bit of each bf16 value (a large sentinel
    for zeros)."""
    b = np.asarray(bits, np.uint16).astype(np.int32)
    ex = (b >> 7) & 0xFF
    m = b & 0x7F
    sig = np.where(ex > 0, m | 0x80, m)
    base = np.where(ex > 0, ex - 134, -133)
    ctz = np.zeros_like(sig)
    s = sig.copy()
    for _ in range(8):
        low = (s & 1) == 0
        grow = low & (s != 0)
        ctz += grow
        s = np.where(grow, s >> 1, s)
    return np.where(sig == 0, 10000, base + ctz).astype(np.int32)


def exactness_margin(x_bits: np.ndarray, w_bits: np.ndarray) -> np.ndarray:
    """Per logit [T, E]: 53 + e - log2(sum |x_i w_i|), e the lowest set bit
    over the nonzero products. Positive: the float64 sum is exact in any
    order. (+inf for a row with no nonzero product.)"""
    lx, lw = lsb_exponents(x_bits), lsb_exponents(w_bits)
    ax = np.abs((np.asarray(x_bits, np.uint16).astype(np.uint32) << 16).view(np.float32)).astype(np.float64)
    aw = np.abs((np.asarray(w_bits, np.uint16).astype(np.uint32) << 16).view(np.float32)).astype(np.float64)
    T, E = lx.shape[0], lw.shape[0]
    emin = np.empty((T, E), np.int64)
    for e in range(E):
        emin[:, e] = (lx + lw[e][None, :]).min(axis=1)
    # sum |p| is a float64 sum of nonnegative terms: relative error < d * 2^-52
    total = (ax @ aw.T) * (1 + x_bits.shape[1] * 2.0 ** -52)
    with np.errstate(divide="ignore"):
        margin = 53 + emin - np.log2(total)
    return np.where(emin >= 5000, np.inf, margin)


def f32_neighbours(v: np.float32):
    """The float32 values next to v, below and above (as exact rationals)."""
    lo = np.nextafter(np.float32(v), np.float32(-np.inf))
    hi = np.nextafter(np.float32(v), np.float32(np.inf))
    return Fraction(float(lo)), Fraction(float(hi))


def rounding_is_order_independent(x_bits: np.ndarray, w_bits: np.ndarray):
    """Per logit: True when every float64 summation of its products (any
    order, any association, with or without fused multiply-adds) rounds to
    the same float32, the correctly rounded one. Either the float64 sum is
    exact (positive margin), or the exact sum lies farther from both
    neighbouring float32 midpoints than the worst-case error of a float64 sum
    of d terms, gamma_(d-1) * sum |p| with gamma_n = n u / (1 - n u),
    u = 2^-53. Returns (ok [T, E], exact [T, E], the smallest ratio of
    midpoint distance to error bound over the logits that are not exact)."""
    m = exactness_margin(x_bits, w_bits)
    exact = m > 0
    ok = exact.copy()
    d = x_bits.shape[1]
    u = Fraction(1, 2 ** 53)
    gamma = (d - 1) * u / (1 - (d - 1) * u)
    worst = None
    for t, e in zip(*np.nonzero(~exact)):
        xs = [bf16_value(b) for b in x_bits[t]]
        ws = [bf16_value(b) for b in w_bits[e]]
        s = sum(a * b for a, b in zip(xs, ws))
        bound = gamma * sum(abs(a * b) for a, b in zip(xs, ws))
        v = round_f32(s)
        lo, hi = f32_neighbours(np.float32(float(v)))
        dist = min(abs(s - (v + lo) / 2), abs(s - (v + hi) / 2))
        ok[t, e] = dist > bound
        r = dist / bound if bound else Fraction(10 ** 9)
        worst = r if worst is None else min(worst, r)
    return ok, exact, (float(worst) if worst is not None else float("inf"))


def engineered(T: int = 48, E: int = 8, d: int = 256, seed: int = 2024):
    """x [T, d], wg [E, d] (bf16 bits) and the correctly rounded logits
    [T, E] (float32), with delta[t, e] in {+1, 0, -1}: the exact dot
    product is the float32 midpoint above its truncation plus delta*2^-40."""
    rng = np.random.default_rng(seed)
    n_corr = 6  # correction terms per expert: base-256 digits of up to 2^47 units
    base = d - n_corr * E
    assert base >= 8
    xf = rng.standard_normal((T, d)).astype(np.float32)
    wf = (rng.standard_normal((E, d)) * 0.02).astype(np.float32)
    # no tiny values: every product a multiple of 2^-38
    xf[np.abs(xf) < 2.0 ** -10] = 0
    wf[np.abs(wf) < 2.0 ** -14] = 0
    x = f32_to_bf16_bits(xf)
    w = f32_to_bf16_bits(wf)
    # cancelling pair: +1024 at the front, -1024 at the back of the random part
    x[:, 0] = bf16_from_dyadic(1, 10)
    x[:, base - 1] = bf16_from_dyadic(1, 10)
    w[:, 0] = W_ONE
    w[:, base - 1] = bf16_from_dyadic(-1, 0)
    # correction block: expert e reads its own n_corr columns with weight 1
    x[:, base:] = 0
    w[:, base:] = 0
    for e in range(E):
        w[e, base + n_corr * e: base + n_corr * (e + 1)] = W_ONE
    # exact sums of the random part: x = X 2^-17 and w = W 2^-21 with integer
    # X, W (no value below 2^-10 resp. 2^-14 is left), so sum x w =
    # (X @ W^T) 2^-38 in exact int64 arithmetic (|X W| < 2^48, d < 2^13 terms)
    assert d < 2 ** 13
    X = np.rint(_bits_to_f64(x[:, :base]) * 2.0 ** 17).astype(np.int64)
    Wi = np.rint(_bits_to_f64(w[:, :base]) * 2.0 ** 21).astype(np.int64)
    assert np.array_equal(X * 2.0 ** -17, _bits_to_f64(x[:, :base]))
    assert np.array_equal(Wi * 2.0 ** -21, _bits_to_f64(w[:, :base]))
    S_int = X @ Wi.T
    expected = np.empty((T, E), np.float32)
    delta = np.empty((T, E), np.int8)
    unit = Fraction(1, 2 ** 40)
    for t in range(T):
        for e in range(E):
            s = Fraction(int(S_int[t, e]), 2 ** 38)
            sign = -1 if s < 0 else 1
            a = abs(s)
            if a < Fraction(1, 16):  # keep ulp/2 a multiple of 2^-40: move the target up
                a += Fraction(1, 4)
            ex = a.numerator.bit_length() - a.denominator.bit_length()
            if Fraction(2) ** ex > a:
                ex -= 1
            ulp = Fraction(2) ** (ex - 23)
            q = int(a // ulp)
            if q >= 2 ** 24 - 1:
                q -= 1
            dl = (t * E + e) % 3 - 1
            target = sign * ((q + Fraction(1, 2)) * ulp + dl * unit)
            n = (target - s) / unit
            assert n.denominator == 1
            n = int(n)
            digits = []
            for _ in range(n_corr):
                r = ((n + 128) % 256) - 128
                digits.append(r)
                n = (n - r) // 256
            assert n == 0
            for j, r in enumerate(digits):
                x[t, base + n_corr * e + j] = bf16_from_dyadic(r, 8 * j - 40) if r else 0
            total = s + sum(Fraction(r) * Fraction(2) ** (8 * j - 40) for j, r in enumerate(digits))
            assert total == target
            expected[t, e] = np.float32(float(round_f32(total)))
            delta[t, e] = dl
    # every logit's float64 sum is exact in any order
    assert (exactness_margin(x, w) > 0).all()
    return x, w, expected, delta
