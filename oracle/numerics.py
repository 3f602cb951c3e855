"""Number formats and exact helpers used by the oracle (test infrastructure).

Nothing here depends on the GPU library.  bf16 tensors are held as uint16 bit
patterns, fp32 tensors as float32 arrays; all arithmetic is float64.
"""
from fractions import Fraction

import numpy as np

BF16_MAX = float((2 - 2.0 ** -7) * 2.0 ** 127)


def bf16_to_f64(bits):
    """Exact value of bf16 bit patterns (uint16 array) as float64."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def f32_to_f64(x):
    return np.asarray(x, dtype=np.float32).astype(np.float64)


def f64_to_f32(x):
    """IEEE round-to-nearest-even float64 -> float32 (one rounding)."""
    return np.asarray(x, dtype=np.float64).astype(np.float32)


def f64_to_bf16(x):
    """Round float64 values to bf16 with ONE round-to-nearest-even step.

    A finite |x| is rounded to the nearest integer multiple of the bf16 unit
    in the last place at its magnitude, 2^(max(floor(log2|x|), -126) - 7),
    ties going to the even multiple; results above the largest finite bf16
    become infinity.  Returns uint16 bit patterns.  (Never goes through a
    float32 rounding first, which would round twice.)
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.zeros(x.shape, dtype=np.uint16)
    sign = np.signbit(x)
    a = np.abs(x)
    nan = np.isnan(x)
    inf = np.isinf(x)
    fin = ~(nan | inf)
    mant, ex = np.frexp(np.where(fin & (a > 0), a, 1.0))  # a = mant * 2^ex, mant in [0.5, 1)
    q = np.maximum(ex - 1, -126) - 7                      # exponent of the bf16 ulp
    r = np.rint(np.ldexp(np.where(fin, a, 0.0), -q))      # nearest multiple, ties to even
    with np.errstate(over="ignore"):
        val = np.ldexp(r, q)                               # may be inf for |x| near the float64 limit
    over = fin & (val > BF16_MAX)
    ok = fin & ~over
    vb = (np.where(ok, val, 0.0).astype(np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    out[ok] = vb[ok]
    out[over | inf] = 0x7F80
    out[nan] = 0x7FC0
    out |= np.where(sign & ~nan, np.uint16(0x8000), np.uint16(0))
    return out


def to_f64(x, dtype):
    """Storage array -> float64 values.  dtype in {"bf16", "f32"}."""
    return bf16_to_f64(x) if dtype == "bf16" else f32_to_f64(x)


def from_f64(x, dtype):
    return f64_to_bf16(x) if dtype == "bf16" else f64_to_f32(x)


def magnitude_key(x, dtype):
    """The bit pattern of |x| in the storage format (an integer, monotone in |x|)."""
    if dtype == "bf16":
        return np.asarray(x, dtype=np.uint16).astype(np.uint32) & np.uint32(0x7FFF)
    return np.asarray(x, dtype=np.float32).view(np.uint32) & np.uint32(0x7FFFFFFF)


def two_sum(a, b):
    """Knuth's error-free transformation: a + b = s + e exactly (float64)."""
    s = a + b
    bb = s - a
    e = (a - (s - bb)) + (b - bb)
    return s, e


def exact_sum_sign(terms):
    """Exact sign (-1, 0, +1) of the real sum of float64 arrays ``terms``.

    Shewchuk's Grow-Expansion (Shewchuk 1997, "Adaptive precision
    floating-point arithmetic and fast robust geometric predicates"): each
    term is added to a nonoverlapping expansion by a chain of two_sum steps;
    the expansion's value equals the real sum exactly, and its sign is the
    sign of its largest-magnitude (last nonzero) component.
    """
    terms = [np.asarray(t, dtype=np.float64) for t in terms]
    exp = []
    for b in terms:
        q = b
        grown = []
        for comp in exp:
            q, h = two_sum(q, comp)
            grown.append(h)
        grown.append(q)
        exp = grown
    sign = np.zeros(terms[0].shape, dtype=np.int8)
    for comp in exp:
        sign = np.where(comp != 0, np.sign(comp).astype(np.int8), sign)
    return sign


def sequential_sum(terms, take=None):
    """float64 sum formed from +0.0 by adding each term in index order.

    With ``take`` (list of boolean arrays), term i is added only where
    take[i] holds.  This fixes the rounding order used for every merged sum.
    """
    acc = np.zeros(np.asarray(terms[0]).shape, dtype=np.float64)
    for i, t in enumerate(terms):
        t = np.asarray(t, dtype=np.float64)
        acc = acc + (t if take is None else np.where(take[i], t, 0.0))
    return acc


def k_from_density(n, rho):
    """Number kept by a density rho over n entries: round(rho*n), halves up.

    ``rho`` may be a Fraction, an int or a decimal string; it is used as an
    exact rational, so e.g. 0.1 * 11534336 = 1153433.6 gives 1153434.
    """
    r = Fraction(rho) if not isinstance(rho, float) else Fraction(repr(rho))
    v = r * n + Fraction(1, 2)
    return int(v.numerator // v.denominator)
