"""Pins for oracle.ties: brute force, invariants, special cases and a hand-worked example."""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import numerics as nm
from oracle import ties

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _store(vals, dtype):
    return nm.from_f64(np.asarray(vals, dtype=np.float64), dtype)


def _brute_topk(vals, k):
    """Pick the largest |x| k times, lowest index first among equals (pure Python)."""
    left = list(range(len(vals)))
    keep = set()
    for _ in range(k):
        best = None
        for i in left:
            if best is None or abs(vals[i]) > abs(vals[best]):
                best = i
        keep.add(best)
        left.remove(best)
    return np.array([i in keep for i in range(len(vals))])


def _tie_heavy(rng, n, dtype):
    v = rng.integers(-6, 7, n).astype(np.float64) * 2.0 ** int(rng.integers(-20, 5))
    v[rng.random(n) < 0.3] = 0.0
    v[rng.random(n) < 0.05] *= -0.0 if dtype == "f32" else 1.0
    if rng.random() < 0.3:
        v[rng.random(n) < 0.1] = 2.0 ** -130 * rng.integers(1, 4)    # subnormals
    return _store(v, dtype)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_topk_matches_pure_python_selection(dtype):
    rng = np.random.default_rng(3)
    for _ in range(60):
        n = int(rng.integers(1, 90))
        x = _tie_heavy(rng, n, dtype)
        k = int(rng.integers(0, n + 1))
        vals = list(nm.to_f64(x, dtype))
        assert np.array_equal(ties.topk_mask(x, k, dtype), _brute_topk(vals, k))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_descriptor_form_equals_sort_form(dtype):
    rng = np.random.default_rng(4)
    for _ in range(200):
        n = int(rng.integers(1, 3000))
        x = _tie_heavy(rng, n, dtype) if rng.random() < 0.7 else _store(rng.standard_normal(n), dtype)
        k = int(rng.integers(0, n + 1))
        d = ties.topk_descriptor(x, k, dtype)
        m = ties.topk_mask(x, k, dtype)
        assert np.array_equal(ties.mask_from_descriptor(x, d, dtype), m)
        if k:
            assert d[1] + d[2] == k and d[2] >= 1


def test_counting_descriptor_equals_brute_force_and_partial_selection():
    """The linear-time counting form (used on the 10^8-10^9-entry tensors of the whole-stack
    checks) gives the partial-selection descriptor and the brute-force mask, ties, zeros,
    subnormals, k = 0, k = N and k > nnz included."""
    rng = np.random.default_rng(14)
    for it in range(300):
        n = int(rng.integers(1, 2500))
        x = _tie_heavy(rng, n, "bf16") if rng.random() < 0.7 else _store(rng.standard_normal(n), "bf16")
        k = int(rng.choice([0, n, int(rng.integers(0, n + 1))]))
        d = ties.topk_descriptor_counting(x, k)
        assert d == ties.topk_descriptor(x, k, "bf16")
        want = _brute_topk(list(nm.to_f64(x, "bf16")), k) if n <= 200 else ties.topk_mask(x, k, "bf16")
        assert np.array_equal(ties.mask_from_descriptor(x, d, "bf16"), want)
    with pytest.raises(FloatingPointError):
        ties.topk_descriptor_counting(np.array([0x3F80, 0x7F80], dtype=np.uint16), 1)
    with pytest.raises(ValueError):
        ties.topk_descriptor_counting(np.zeros(4, dtype=np.uint16), 5)


def test_topk_invariants_and_scale_invariance():
    rng = np.random.default_rng(5)
    for _ in range(50):
        n = 4096
        x = _tie_heavy(rng, n, "bf16")
        k = int(rng.integers(1, n))
        m = ties.topk_mask(x, k, "bf16")
        key = nm.magnitude_key(x, "bf16").astype(np.int64)
        assert m.sum() == k
        assert key[m].min() >= key[~m].max()
        t = key[m].min()
        if (key[~m] == t).any():
            assert np.flatnonzero(m & (key == t)).max() < np.flatnonzero(~m & (key == t)).min()
        xs = _store(nm.to_f64(x, "bf16") * 2.0 ** 7, "bf16")
        assert np.array_equal(ties.topk_mask(xs, k, "bf16"), m)


def test_descriptor_k_zero_and_full():
    x = _store([0.5, -0.0, 0.0, 2.0], "bf16")
    assert ties.topk_descriptor(x, 0, "bf16") == (0xFFFFFFFF, 0, 0, 0)
    d = ties.topk_descriptor(x, 4, "bf16")
    assert d[0] == 0 and d[1] == 2 and d[2] == 2 and d[3] == 4        # whole zero bucket kept: cutoff = N
    d = ties.topk_descriptor(x, 3, "bf16")           # k > nnz: the lowest-index zero is kept
    assert d == (0, 2, 1, 2)
    with pytest.raises(ValueError):
        ties.topk_descriptor(x, 5, "bf16")


def _fr(s):
    return Fraction(s)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_hand_worked_example(dtype):
    g = json.load(open(os.path.join(GOLD, "ties_worked_example.json")))
    base = _store(g["base"], dtype)
    deltas = [_store(d, dtype) for d in g["deltas"]]
    r = ties.merge_unit(base, deltas, dtype, "ties", k=g["k"])
    assert [list(m.astype(int)) for m in r["masks"]] == g["masks"]
    assert list(r["gamma"]) == g["gamma"]
    assert [Fraction(float(v)) for v in r["u"]] == [_fr(s) for s in g["ties_tau"]]
    assert np.array_equal(r["out"], _store([float(_fr(s)) for s in g["ties_out_lambda_1"]], dtype))
    r = ties.merge_unit(base, deltas, dtype, "ties", k=g["k"], lam=0.5)
    assert np.array_equal(r["out"], _store([float(_fr(s)) for s in g["ties_out_lambda_half"]], dtype))
    r = ties.merge_unit(base, deltas, dtype, "ta")
    assert np.array_equal(r["out"], _store([float(_fr(s)) for s in g["ta_out_lambda_1"]], dtype))
    r = ties.merge_unit(base, deltas, dtype, "ram", eps=g["ram_eps"])
    for got, s in zip(r["u"], g["ram_tau"]):
        assert abs(Fraction(float(got)) - _fr(s)) <= Fraction(1, 2 ** 54)


def _rand_unit(rng, n, K, dtype, p_zero=0.5, scale=1e-3):
    base = _store(rng.standard_normal(n) * 0.02, dtype)
    ds = []
    for _ in range(K):
        v = rng.standard_normal(n) * scale
        v[rng.random(n) < p_zero] = 0.0
        ds.append(_store(v, dtype))
    return base, ds


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_k1_merge_is_identity_on_masked_delta(dtype):
    rng = np.random.default_rng(6)
    base, ds = _rand_unit(rng, 5000, 1, dtype)
    k = 700
    r = ties.merge_unit(base, ds, dtype, "ties", k=k)
    m = ties.topk_mask(ds[0], k, dtype)
    assert np.array_equal(r["u"], np.where(m, nm.to_f64(ds[0], dtype), 0.0))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_identical_experts_give_masked_delta(dtype):
    rng = np.random.default_rng(7)
    base, ds = _rand_unit(rng, 5000, 1, dtype)
    r = ties.merge_unit(base, ds * 3, dtype, "ties", k=900)
    m = ties.topk_mask(ds[0], 900, dtype)
    assert np.array_equal(r["u"], np.where(m, nm.to_f64(ds[0], dtype), 0.0))


def test_opposite_experts_cancel():
    rng = np.random.default_rng(8)
    base, ds = _rand_unit(rng, 5000, 1, "bf16")
    neg = (ds[0] ^ np.uint16(0x8000)).astype(np.uint16)
    r = ties.merge_unit(base, [ds[0], neg], "bf16", "ties", k=1200)
    assert np.all(r["gamma"] == 0)
    assert np.array_equal(r["out"], nm.from_f64(nm.to_f64(base, "bf16") + 0.0, "bf16"))


def test_full_density_same_sign_is_mean_of_nonzeros_and_ram_eps0():
    rng = np.random.default_rng(9)
    n, K = 3000, 4
    vals = np.abs(rng.standard_normal((K, n))) * 1e-3 * np.sign(rng.standard_normal(n))
    vals[rng.random((K, n)) < 0.4] = 0.0
    ds = [_store(v, "f32") for v in vals]
    base = _store(np.zeros(n), "f32")
    r = ties.merge_unit(base, ds, "f32", "ties", k=n)
    x = nm.to_f64(np.stack(ds), "f32")
    cnt = (x != 0).sum(0)
    mean = np.where(cnt > 0, nm.sequential_sum(list(x)) / np.maximum(cnt, 1), 0.0)
    assert np.array_equal(r["u"], mean)
    r2 = ties.merge_unit(base, ds, "f32", "ram", eps=0.0)
    assert np.array_equal(r2["u"], mean)


def test_lambda_zero_returns_base():
    rng = np.random.default_rng(10)
    base, ds = _rand_unit(rng, 4000, 3, "bf16")
    r = ties.merge_unit(base, ds, "bf16", "ties", k=500, lam=0.0)
    w = nm.to_f64(base, "bf16")
    assert np.array_equal(r["out"], nm.from_f64(w + 0.0, "bf16"))


def test_power_of_two_scaling_equivariance():
    rng = np.random.default_rng(11)
    base, ds = _rand_unit(rng, 4000, 4, "bf16")
    r = ties.merge_unit(base, ds, "bf16", "ties", k=600)
    ds2 = [_store(nm.to_f64(d, "bf16") * 2.0 ** -9, "bf16") for d in ds]
    r2 = ties.merge_unit(base, ds2, "bf16", "ties", k=600)
    assert np.array_equal(r2["u"], r["u"] * 2.0 ** -9)


def test_expert_order_symmetry():
    rng = np.random.default_rng(12)
    base, ds = _rand_unit(rng, 4000, 4, "bf16")
    r = ties.merge_unit(base, ds, "bf16", "ties", k=800)
    r2 = ties.merge_unit(base, ds[::-1], "bf16", "ties", k=800)
    assert np.array_equal(r["gamma"], r2["gamma"])
    assert np.array_equal(r["u"], r2["u"])     # exact sums: the span of these values is small


def test_ta_lambda_one_over_k_is_the_1d_average():
    from oracle.spectral import average_1d
    rng = np.random.default_rng(13)
    for K in (2, 4):
        base, ds = _rand_unit(rng, 3000, K, "f32")
        r = ties.merge_unit(base, ds, "f32", "ta", lam=1.0 / K)
        w0 = nm.to_f64(base, "f32")
        avg = average_1d(w0, [w0 + nm.to_f64(d, "f32") for d in ds])
        assert np.allclose(w0 + r["u"], avg, rtol=0, atol=1e-15)


def test_merge_at_matches_whole_unit():
    rng = np.random.default_rng(14)
    base, ds = _rand_unit(rng, 20000, 4, "bf16")
    k = 2100
    whole = ties.merge_unit(base, ds, "bf16", "ties", k=k)
    descs = [ties.topk_descriptor(d, k, "bf16") for d in ds]
    idx = np.sort(rng.choice(20000, 500, replace=False))
    part = ties.merge_at(base[idx], [d[idx] for d in ds], "ties", descs, idx, "bf16")
    assert np.array_equal(part["out"], whole["out"][idx])
    assert np.array_equal(part["gamma"], whole["gamma"][idx])


def test_nonfinite_input_raises():
    x = _store([1.0, np.nan], "f32")
    with pytest.raises(FloatingPointError):
        ties.topk_mask(x, 1, "f32")
    with pytest.raises(FloatingPointError):
        ties.merge_unit(x, [x], "f32", "ta")


def _brute_joint(pieces, k):
    """Joint TopKMask by repeated maximum over (|x| desc, piece, index) in pure Python."""
    items = [(abs(v), p, i) for p, vals in enumerate(pieces) for i, v in enumerate(vals)]
    left = list(range(len(items)))
    keep = set()
    for _ in range(k):
        best = None
        for q in left:
            a, p, i = items[q]
            if best is None or a > items[best][0]:
                best = q
        keep.add(best)
        left.remove(best)
    out = [np.zeros(len(v), dtype=bool) for v in pieces]
    for q in keep:
        _, p, i = items[q]
        out[p][i] = True
    return out


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_joint_topk_matches_pure_python_selection(dtype):
    """Ties across pieces go to the earlier piece, then the lower index; k spans pieces."""
    rng = np.random.default_rng(8)
    lens = [7, 1, 12, 0, 9]
    pieces_f = [list(rng.choice([0.0, 0.5, -0.5, 1.0, -2.0, 0.25], size=n)) for n in lens]
    pieces = [_store(v, dtype) for v in pieces_f]
    vals = [list(nm.to_f64(p, dtype)) for p in pieces]
    for k in (0, 1, 5, 13, 20, sum(lens)):
        got = ties.topk_mask_joint(pieces, k, dtype)
        want = _brute_joint(vals, k)
        assert all(np.array_equal(g, w) for g, w in zip(got, want)), k
        assert sum(int(g.sum()) for g in got) == k


def test_joint_topk_of_one_piece_is_topk():
    rng = np.random.default_rng(9)
    d = _store(rng.standard_normal(300) * 1e-3, "bf16")
    for k in (0, 17, 300):
        assert np.array_equal(ties.topk_mask_joint([d], k, "bf16")[0], ties.topk_mask(d, k, "bf16"))
