"""Pins for oracle.numerics against brute force and exact rational arithmetic."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import numerics as nm


def _all_bf16_finite():
    bits = np.arange(0, 0x7F80, dtype=np.uint32).astype(np.uint16)      # +0 .. largest finite
    vals = nm.bf16_to_f64(bits)
    return bits, vals


def _brute_bf16(x):
    """Nearest finite bf16 by exhaustive search over all patterns, ties to even pattern."""
    bits, vals = _all_bf16_finite()
    a = abs(x)
    fa = Fraction(a)
    i = int(np.searchsorted(vals, a))
    cands = [j for j in (i - 1, i, i + 1) if 0 <= j < vals.size]
    best = None
    for j in cands:
        dist = abs(Fraction(float(vals[j])) - fa)
        key = (dist, int(bits[j]) & 1)
        if best is None or key < best[0]:
            best = (key, int(bits[j]))
    res = best[1]
    # beyond the largest finite value: round to infinity once past the midpoint to 2^128
    top = Fraction(float(vals[-1]))
    mid = top + (Fraction(2) ** 128 - top) / 2
    if fa >= mid:
        res = 0x7F80
    if np.signbit(x):
        res |= 0x8000
    return res


def test_bf16_decode_known_patterns():
    got = nm.bf16_to_f64(np.array([0x3F80, 0xC000, 0x0001, 0x7F7F, 0x8000, 0x0080], dtype=np.uint16))
    assert got[0] == 1.0 and got[1] == -2.0 and got[2] == 2.0 ** -133
    assert got[3] == (2 - 2.0 ** -7) * 2.0 ** 127 and got[4] == 0.0 and np.signbit(got[4])
    assert got[5] == 2.0 ** -126


def test_f64_to_bf16_brute_force_random():
    rng = np.random.default_rng(0)
    xs = np.concatenate([
        rng.standard_normal(300) * 10.0 ** rng.integers(-45, 39, 300),
        rng.standard_normal(100) * 1e-39,              # bf16 subnormal range
        rng.standard_normal(50) * 1e-41,
    ])
    got = nm.f64_to_bf16(xs)
    for x, g in zip(xs, got):
        assert int(g) == _brute_bf16(float(x)), x


def test_f64_to_bf16_midpoints_and_edges():
    bits, vals = _all_bf16_finite()
    rng = np.random.default_rng(1)
    pick = rng.integers(0, vals.size - 1, 400)
    lo, hi = vals[pick], vals[pick + 1]
    mids = (lo + hi) / 2                       # exact midpoints (representable in float64)
    got = nm.f64_to_bf16(mids)
    for m, l, g in zip(mids, pick, got):
        even = l if (int(bits[l]) & 1) == 0 else l + 1
        assert int(g) == int(bits[even]), m
        assert int(g) == _brute_bf16(float(m))
    # just above / below a midpoint
    for m in mids[:50]:
        assert int(nm.f64_to_bf16(np.array([np.nextafter(m, np.inf)]))[0]) == _brute_bf16(float(np.nextafter(m, np.inf)))
        assert int(nm.f64_to_bf16(np.array([np.nextafter(m, -np.inf)]))[0]) == _brute_bf16(float(np.nextafter(m, -np.inf)))
    top = float(vals[-1])
    assert nm.f64_to_bf16(np.array([top, -top]))[0] == 0x7F7F
    assert nm.f64_to_bf16(np.array([2.0 ** 128]))[0] == 0x7F80
    assert nm.f64_to_bf16(np.array([1e300, -np.inf, np.inf]))[1] == 0xFF80
    assert nm.f64_to_bf16(np.array([2.0 ** -134]))[0] == 0          # half of the smallest subnormal: tie to even 0
    assert nm.f64_to_bf16(np.array([3 * 2.0 ** -135]))[0] == 1
    z = nm.f64_to_bf16(np.array([-0.0, 0.0]))
    assert z[0] == 0x8000 and z[1] == 0


def test_f64_to_bf16_single_rounding_differs_from_double_rounding():
    # x just above a bf16 midpoint but within half an fp32 ulp of it: rounding via fp32 lands on
    # the midpoint and then ties to even (down); the single rounding must go up.
    lo = 1.0
    mid = 1.0 + 2.0 ** -8
    x = mid + 2.0 ** -30
    via_f32 = np.float32(x).view(np.uint32)
    assert float(np.float32(x)) == mid
    assert (int(via_f32) >> 16) == 0x3F80
    assert int(nm.f64_to_bf16(np.array([x]))[0]) == 0x3F81
    assert lo < x


def test_exact_sum_sign_against_fractions():
    rng = np.random.default_rng(2)
    for trial in range(300):
        K = int(rng.integers(1, 7))
        n = 64
        ex = rng.integers(-140, 120, size=(K, n))
        v = rng.standard_normal((K, n)) * np.exp2(ex.astype(np.float64))
        v = nm.bf16_to_f64(nm.f64_to_bf16(v)) if trial % 2 else v.astype(np.float32).astype(np.float64)
        if trial % 5 == 0:        # force exact cancellations
            v[-1] = -np.sum(v[:-1], axis=0) if K > 1 else v[-1]
            v[-1] = nm.bf16_to_f64(nm.f64_to_bf16(v[-1]))
        got = nm.exact_sum_sign(list(v))
        for p in range(n):
            s = sum(Fraction(float(v[i, p])) for i in range(K))
            assert got[p] == (s > 0) - (s < 0)


def test_exact_sum_sign_beats_naive_order():
    a = np.array([1.0]); b = np.array([1e-30]); c = np.array([-1.0])
    assert ((a + b) + c)[0] == 0.0
    assert nm.exact_sum_sign([a, b, c])[0] == 1
    assert nm.exact_sum_sign([np.array([0.0]), np.array([-0.0])])[0] == 0


@pytest.mark.parametrize("n,rho,k", [(65536, "0.2", 13107), (2048 * 5632, "0.1", 1153434),
                                     (2048 * 2048, "0.1", 419430), (18944 * 3584, "0.1", 6789530),
                                     (152064 * 3584, "0.1", 54499738), (1536 * 1536, "0.05", 117965),
                                     (5, "0.1", 1), (15, "0.1", 2), (25, "0.1", 3), (10, "0", 0), (7, "1", 7)])
def test_k_from_density(n, rho, k):
    assert nm.k_from_density(n, rho) == k
