"""GPU parity of the single-read bf16 TIES path (iso_update, FUSED, TIES, desc NULL).

That path brackets each delta's TopKMask threshold from a sampled key histogram, merges
every coordinate once and fixes up the coordinates whose keys fell inside the bracket.  A
tensor it cannot settle (misleading sample, bracket too wide, record region full) takes
the exact two-pass path on the device.  Either way the result must equal the oracle's bit
for bit; the fallback count says which route a tensor took, so each route is exercised on
purpose here.  Deltas above 2^20 entries are sampled (4096 blocks of 256 entries at
floor(b * nb / 4096), nb = n / 256); smaller ones are histogrammed whole.
"""
import numpy as np
import pytest

from oracle import numerics as nm
from oracle import ties

import paper_2607_19331_amd as iso
from tests.gpu_helpers import Unit, from_dev, say

pytestmark = pytest.mark.gpu


def fused(units, K, lam=1.0, want_sign=True):
    import torch
    es = [u.entry() for u in units]
    ws = iso.workspace(iso.OP_UPDATE_FUSED_SELECT, es, K, iso.BF16)
    signs = [torch.empty(max(u.n, 16), dtype=torch.int8, device="cuda") for u in units] if want_sign else None
    iso.iso_update(es, K, iso.BF16, iso.UPDATE_FUSED, merge=iso.MERGE_TIES, lam=lam, desc=None, sign_out=signs,
                   ws=ws)
    st = iso.iso_read_device_status(ws)
    fb = iso.iso_read_fallback_count(ws)
    outs = [from_dev(u.dout, u.n, "bf16") for u in units]
    sg = [s.cpu().numpy()[:u.n] for s, u in zip(signs, units)] if want_sign else None
    return outs, sg, st, fb


def check(units, K, outs, sg, lam=1.0):
    for j, u in enumerate(units):
        if not u.n:
            continue
        r = ties.merge_unit(u.base, u.deltas, "bf16", "ties", k=u.k, lam=lam)
        assert np.array_equal(outs[j], r["out"]), j
        if sg is not None:
            assert np.array_equal(sg[j], r["gamma"]), j


def normal_unit(rng, rows, cols, K, rho=0.1, p_zero=0.5, scale=1e-3, k=None):
    n = rows * cols
    base = nm.from_f64(rng.standard_normal(n) * 0.02, "bf16")
    ds = []
    for _ in range(K):
        v = rng.standard_normal(n) * scale
        v[rng.random(n) < p_zero] = 0.0
        ds.append(nm.from_f64(v, "bf16"))
    if k is None:
        k = nm.k_from_density(n, rho)
    return Unit(rows, cols, base, ds, "bf16", k)


def test_sampled_and_exact_tensors_settle_in_one_read():
    rng = np.random.default_rng(101)
    units = [normal_unit(rng, 2048, 4096, 4),                 # sampled
             normal_unit(rng, 2049, 1025, 4, rho=0.3),        # sampled, ragged (n % 8 != 0)
             normal_unit(rng, 512, 3584, 4),                  # sampled, just above 2^20 entries
             normal_unit(rng, 1024, 1024, 4),                 # whole-delta histogram (2^20 entries)
             normal_unit(rng, 3, 5, 4)]
    say("fused single read: 2048x4096, 2049x1025, 512x3584, 1024x1024, 3x5, K=4")
    outs, sg, st, fb = fused(units, 4)
    assert st == 0
    assert fb == 0
    check(units, 4, outs, sg)


def test_lambda_and_k_extremes():
    rng = np.random.default_rng(102)
    n1 = 1024 * 4096
    units = [normal_unit(rng, 1024, 4096, 3, k=0),
             normal_unit(rng, 1024, 4096, 3, k=n1),
             normal_unit(rng, 1024, 4096, 3, rho=0.7),        # threshold among the zeros: every nonzero kept
             normal_unit(rng, 300, 301, 3, k=300 * 301),
             normal_unit(rng, 300, 301, 3, k=0)]
    say("fused k = 0, k = n, rho 0.7, lambda 0.5, K=3")
    outs, sg, st, fb = fused(units, 3, lam=0.5)
    assert st == 0
    assert fb == 0
    check(units, 3, outs, sg, lam=0.5)


def test_misleading_sample_takes_the_two_pass_path():
    """Every 4th 256-entry block (the sampled ones at this size) holds tiny values, the
    others large ones: the sample brackets the threshold far too low."""
    rng = np.random.default_rng(103)
    rows, cols, K = 1024, 4096, 2
    n = rows * cols
    blk = (np.arange(n) // 256) % 4 == 0
    base = nm.from_f64(rng.standard_normal(n) * 0.02, "bf16")
    ds = []
    for _ in range(K):
        v = rng.standard_normal(n) * np.where(blk, 1e-6, 1e-2)
        ds.append(nm.from_f64(v, "bf16"))
    bad = Unit(rows, cols, base, ds, "bf16", nm.k_from_density(n, 0.1))
    good = normal_unit(rng, 1024, 4096, K)
    say("fused misleading sample 1024x4096 K=2 + a normal tensor")
    outs, sg, st, fb = fused([good, bad], K)
    assert st == 0
    assert fb == 1
    check([good, bad], K, outs, sg)


def test_tiny_k_bracket_too_wide_takes_the_two_pass_path():
    rng = np.random.default_rng(104)
    u = normal_unit(rng, 1024, 4096, 2, k=10)
    say("fused k = 10 on 1024x4096")
    outs, sg, st, fb = fused([u], 2)
    assert st == 0
    assert fb == 1
    check([u], 2, outs, sg)


def test_heavy_ties_fill_the_record_region():
    """Eleven distinct magnitudes: the threshold code holds about a fifth of the entries,
    more than the record regions can hold."""
    rng = np.random.default_rng(105)
    rows, cols, K = 256, 1000, 3
    n = rows * cols
    base = nm.from_f64(rng.standard_normal(n) * 0.02, "bf16")
    ds = [nm.from_f64(rng.integers(-5, 6, n).astype(np.float64) * 2.0 ** -12, "bf16") for _ in range(K)]
    u = Unit(rows, cols, base, ds, "bf16", nm.k_from_density(n, 0.3))
    v = normal_unit(rng, 256, 1000, K)
    say("fused heavy ties 256x1000 K=3 + a normal tensor")
    outs, sg, st, fb = fused([u, v], K)
    assert st == 0
    assert fb == 1
    check([u, v], K, outs, sg)


@pytest.mark.parametrize("K", [1, 2, 5, 8])
def test_other_expert_counts(K):
    rng = np.random.default_rng(110 + K)
    units = [normal_unit(rng, 1536, 2048, K, rho=0.2), normal_unit(rng, 77, 1001, K)]
    say(f"fused K={K} 1536x2048 + 77x1001")
    outs, sg, st, fb = fused(units, K)
    assert st == 0
    assert fb == 0
    check(units, K, outs, sg)


def test_repeat_calls_reuse_the_workspace():
    """Second call on the same workspace with other data: no state may leak between calls."""
    import torch
    rng = np.random.default_rng(120)
    a = [normal_unit(rng, 1024, 4096, 2), normal_unit(rng, 100, 100, 2)]
    b = [normal_unit(rng, 1024, 4096, 2, rho=0.05), normal_unit(rng, 100, 100, 2, rho=0.5)]
    es_a = [u.entry() for u in a]
    ws = iso.workspace(iso.OP_UPDATE_FUSED_SELECT, es_a, 2, iso.BF16)
    say("fused repeat on one workspace")
    for units in (a, b, a):
        es = [u.entry() for u in units]
        iso.iso_update(es, 2, iso.BF16, iso.UPDATE_FUSED, merge=iso.MERGE_TIES, desc=None, ws=ws)
        assert iso.iso_read_device_status(ws) == 0
        outs = [from_dev(u.dout, u.n, "bf16") for u in units]
        check(units, 2, outs, None)
    torch.cuda.synchronize()


@pytest.mark.parametrize("want_sign", [False, True], ids=["no_sign", "sign"])
def test_binary32_midpoints_take_the_exact_rounding(want_sign):
    """Dense deltas (every entry kept) and lambda = 0.3 put a few dozen results of a 4M-entry
    tensor on a bf16 midpoint once rounded to binary32 (low half 0x8000) while the binary64
    value is not one; rounding the binary32 value again would miss the correct bf16 in about
    half of them.  The pass redoes those pairs with round-to-odd: bit-exact with the oracle."""
    rng = np.random.default_rng(3)
    R, C, K, lam = 2048, 2048, 3, 0.3
    n = R * C
    base = nm.from_f64(rng.standard_normal(n) * 0.02, "bf16")
    ds = [nm.from_f64(rng.standard_normal(n) * 1e-3, "bf16") for _ in range(K)]
    u = Unit(R, C, base, ds, "bf16", n)
    ref = ties.merge_unit(base, ds, "bf16", "ties", k=n, lam=lam)
    v = nm.to_f64(base, "bf16") + ref["u"]
    f = v.astype(np.float32)
    mid = ((f.view(np.uint32) & 0xFFFF) == 0x8000) & (f.astype(np.float64) != v)
    assert mid.sum() >= 16
    assert np.any(nm.f64_to_bf16(f.astype(np.float64)) != ref["out"])   # the case is not vacuous
    say(f"fused bf16 midpoints: {int(mid.sum())} binary32 midpoints, sign output {want_sign}")
    outs, sg, st, fb = fused([u], K, lam=lam, want_sign=want_sign)
    assert st == 0 and fb == 0
    assert np.array_equal(outs[0], ref["out"])
    if want_sign:
        assert np.array_equal(sg[0], ref["gamma"])


def test_cancelling_base_takes_the_exact_rounding():
    """A base that nearly cancels the merged update (w0 = -bf16(lambda tau)): results far below
    the base's magnitude, where any shortcut in the binary64 sequence would show; bit-exact with
    the oracle, lambda 1 and 0.3."""
    rng = np.random.default_rng(4)
    R, C, K = 512, 512, 3
    n = R * C
    ds = [nm.from_f64(rng.standard_normal(n) * 1e-3, "bf16") for _ in range(K)]
    for lam in (1.0, 0.3):
        probe = ties.merge_unit(nm.from_f64(np.zeros(n), "bf16"), ds, "bf16", "ties", k=n, lam=lam)
        base = nm.f64_to_bf16(-probe["u"])
        u = Unit(R, C, base, ds, "bf16", n)
        ref = ties.merge_unit(base, ds, "bf16", "ties", k=n, lam=lam)
        w0 = np.abs(nm.to_f64(base, "bf16"))
        assert np.mean(w0 > 16 * np.abs(nm.to_f64(ref["out"], "bf16"))) > 0.5   # mostly cancelling
        say(f"fused cancelling base, lambda {lam}")
        outs, sg, st, fb = fused([u], K, lam=lam, want_sign=False)
        assert st == 0 and fb == 0
        assert np.array_equal(outs[0], ref["out"])
