"""GPU parity of the element-wise path against the CPU oracle, bit for bit.

Descriptors, masks and elected signs are integer results and must match exactly; the
merged values follow the same binary64 sequence as the oracle, so they must match
exactly too (stricter than the 1e-6 relative / 1 bf16 ulp acceptance bound).
"""
import numpy as np
import pytest

from oracle import numerics as nm
from oracle import ties

pytestmark = pytest.mark.gpu

from tests.gpu_helpers import (Unit, bits_to_mask, run_apply, run_fused, run_merge, run_sign, run_topk, say)  # noqa: E402


def _store(v, dtype):
    return nm.from_f64(np.asarray(v, dtype=np.float64), dtype)


def make_unit(rng, rows, cols, K, dtype, kind, rho=0.2):
    n = rows * cols
    base = _store(rng.standard_normal(n) * 0.02, dtype)
    ds = []
    for i in range(K):
        if kind == "rand":
            v = rng.standard_normal(n) * 1e-3
            v[rng.random(n) < 0.6] = 0.0
        elif kind == "ties":
            v = rng.integers(-5, 6, n).astype(np.float64) * 2.0 ** -12
            v[rng.random(n) < 0.2] = 0.0
            v[rng.random(n) < 0.05] = -0.0
            if n:
                v[rng.random(n) < 0.02] = 2.0 ** -130 * rng.integers(1, 4)
        elif kind == "span":
            e = rng.integers(-60, 10, n).astype(np.float64)
            v = rng.standard_normal(n) * 2.0 ** e
            v[rng.random(n) < 0.3] = 0.0
        elif kind == "cancel":
            v = rng.standard_normal(n) * 1e-3
            if i % 2 == 1:
                v = -nm.to_f64(ds[-1], dtype)           # exact cancellation with the previous expert
        else:
            raise ValueError(kind)
        ds.append(_store(v, dtype))
    k = nm.k_from_density(n, rho) if n else 0
    return Unit(rows, cols, base, ds, dtype, k)


CASES = [
    ("f32", 3, "rand", [(256, 256)]),
    ("bf16", 4, "rand", [(256, 256), (37, 53), (1, 1), (1, 7), (0, 5), (3, 4099)]),
    ("bf16", 2, "ties", [(64, 1000), (5, 9)]),
    ("f32", 2, "ties", [(64, 1000), (13, 17)]),
    ("bf16", 4, "span", [(128, 257)]),
    ("f32", 3, "span", [(100, 101)]),
    ("bf16", 4, "cancel", [(64, 512)]),
    ("bf16", 1, "rand", [(50, 77)]),
    ("bf16", 8, "rand", [(40, 300)]),
    ("f32", 5, "ties", [(33, 129)]),
]


def _ids(c):
    return f"{c[0]}-K{c[1]}-{c[2]}-{'x'.join(str(r) + '_' + str(cc) for r, cc in c[3])}"


@pytest.fixture(scope="module")
def cases():
    rng = np.random.default_rng(1234)
    out = {}
    for c in CASES:
        dtype, K, kind, shapes = c
        out[_ids(c)] = (dtype, K, kind, [make_unit(rng, r, cc, K, dtype, kind) for r, cc in shapes])
    return out


@pytest.mark.parametrize("case", [_ids(c) for c in CASES])
def test_topk_descriptors_and_masks(cases, case):
    dtype, K, kind, units = cases[case]
    say(f"topk {case}")
    d, bits, st, _ = run_topk(units, K, dtype, with_bits=True)
    assert st == 0
    for j, u in enumerate(units):
        for i in range(K):
            want = ties.topk_descriptor(u.deltas[i], u.k, dtype)
            got = d[j * K + i]
            assert (got[0], got[2], got[3], got[4]) == want, (j, i, got, want)
            if u.n:
                assert got[1] == int(nm.magnitude_key(u.deltas[i], dtype).max())
                m = bits_to_mask(bits[j * K + i], u.n)
                assert np.array_equal(m, ties.topk_mask(u.deltas[i], u.k, dtype))


@pytest.mark.parametrize("case", [_ids(c) for c in CASES])
def test_sign_and_merge_and_fused(cases, case):
    dtype, K, kind, units = cases[case]
    say(f"sign/merge/fused {case}")
    _, _, st, desc = run_topk(units, K, dtype)
    assert st == 0
    refs = [ties.merge_unit(u.base, u.deltas, dtype, "ties", k=u.k) if u.n else None for u in units]
    signs, st = run_sign(units, K, dtype, desc)
    assert st == 0
    taus, st = run_merge(units, K, dtype, 1, desc)
    assert st == 0
    outs, fs, st = run_fused(units, K, dtype, 1, desc=desc, want_sign=True)
    assert st == 0
    outs2, _, st = run_fused(units, K, dtype, 1, desc=None)
    assert st == 0
    for j, u in enumerate(units):
        if not u.n:
            continue
        r = refs[j]
        assert np.array_equal(signs[j], r["gamma"]), j
        assert np.array_equal(fs[j], r["gamma"]), j
        assert np.array_equal(taus[j].view(np.uint32), r["tau"].view(np.uint32)), j
        assert np.array_equal(outs[j].view(np.uint8), r["out"].view(np.uint8)), j
        assert np.array_equal(outs2[j].view(np.uint8), r["out"].view(np.uint8)), j


@pytest.mark.parametrize("case", [_ids(c) for c in CASES])
def test_ta_ram_apply(cases, case):
    dtype, K, kind, units = cases[case]
    say(f"ta/ram/apply {case}")
    for mode, name, lam, eps in [(0, "ta", 1.0, 0.0), (0, "ta", 0.25, 0.0), (2, "ram", 1.0, 1e-5),
                                 (2, "ram", 1.0, 0.0)]:
        outs, _, st = run_fused(units, K, dtype, mode, lam=lam, eps=eps)
        assert st == 0
        taus, st = run_merge(units, K, dtype, mode, None, lam=lam, eps=eps)
        assert st == 0
        for j, u in enumerate(units):
            if not u.n:
                continue
            r = ties.merge_unit(u.base, u.deltas, dtype, name, lam=lam, eps=eps)
            assert np.array_equal(outs[j].view(np.uint8), r["out"].view(np.uint8)), (name, j)
            assert np.array_equal(taus[j].view(np.uint32), r["tau"].view(np.uint32)), (name, j)
    rng = np.random.default_rng(5)
    thost = [(rng.standard_normal(u.n) * 1e-3).astype(np.float32) for u in units]
    outs, st = run_apply(units, dtype, thost, lam=0.5)
    assert st == 0
    for j, u in enumerate(units):
        if u.n:
            want = ties.apply_update(u.base, 0.5 * thost[j].astype(np.float64), dtype)
            assert np.array_equal(outs[j].view(np.uint8), want.view(np.uint8))


def test_lambda_variants_and_unmasked_sign():
    rng = np.random.default_rng(7)
    u = make_unit(rng, 96, 333, 3, "bf16", "rand")
    say("lambda variants bf16 96x333 K=3")
    _, _, st, desc = run_topk([u], 3, "bf16")
    for lam in (0.0, 0.5, -1.0, 3.0):
        outs, _, st = run_fused([u], 3, "bf16", 1, desc=desc, lam=lam)
        assert st == 0
        r = ties.merge_unit(u.base, u.deltas, "bf16", "ties", k=u.k, lam=lam)
        assert np.array_equal(outs[0], r["out"]), lam
    signs, st = run_sign([u], 3, "bf16", None)
    xs = [nm.to_f64(d, "bf16") for d in u.deltas]
    assert np.array_equal(signs[0], nm.exact_sum_sign(xs))


def test_nonfinite_is_reported():
    rng = np.random.default_rng(8)
    u = make_unit(rng, 32, 64, 2, "bf16", "rand")
    bad = u.deltas[1].copy()
    bad[100] = 0x7FC0          # NaN
    u2 = Unit(32, 64, u.base, [u.deltas[0], bad], "bf16", u.k)
    say("nonfinite delta")
    _, _, st, _ = run_topk([u2], 2, "bf16")
    assert st == 4
    outs, _, st = run_fused([u2], 2, "bf16", 0)
    assert st == 4
    b = u.base.copy()
    b[5] = 0x7F80              # +inf in the base
    u3 = Unit(32, 64, b, u.deltas, "bf16", u.k)
    outs, _, st = run_fused([u3], 2, "bf16", 1)
    assert st == 4
    outs, _, st = run_fused([u], 2, "bf16", 1)
    assert st == 0


def test_repeat_runs_are_bitwise_identical():
    rng = np.random.default_rng(9)
    units = [make_unit(rng, 200, 300, 4, "bf16", "ties"), make_unit(rng, 100, 1000, 4, "bf16", "rand")]
    say("determinism")
    a, _, _ = run_fused(units, 4, "bf16", 1)
    b, _, _ = run_fused(units, 4, "bf16", 1)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
