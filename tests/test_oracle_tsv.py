"""Pins for oracle.tsv (TSV-Merge, App. F)."""
import math

import numpy as np

from oracle import numerics as nm
from oracle import tsv


def test_closed_form_two_rank_one_deltas():
    """Delta_1 = a e1 e1^T, Delta_2 = b u2 e2^T with u2 at angle phi.  U = [e1 u2] has polar factor with
    columns at angles phi/2 -+ pi/4 (the orthonormal pair nearest to U, symmetric about the bisector);
    V = I.  So Delta_hat = [[a cos p1, b cos p2], [a sin p1, b sin p2]], p1,2 = phi/2 -+ pi/4."""
    for a, b, phi in [(2.0, 1.0, 0.7), (1.0, 3.0, 1.2), (0.5, 0.5, math.pi / 2)]:
        d1 = np.array([[a, 0.0], [0.0, 0.0]])
        d2 = b * np.outer([math.cos(phi), math.sin(phi)], [0.0, 1.0])
        dh, _ = tsv.tsv_delta([d1, d2], 1)
        p1, p2 = phi / 2 - math.pi / 4, phi / 2 + math.pi / 4
        want = np.array([[a * math.cos(p1), b * math.cos(p2)], [a * math.sin(p1), b * math.sin(p2)]])
        assert np.allclose(dh, want, atol=1e-14)


def test_single_delta_is_best_rank_r():
    rng = np.random.default_rng(0)
    d = rng.standard_normal((50, 40))
    s = np.linalg.svd(d, compute_uv=False)
    for r in (1, 5, 20):
        dh, _ = tsv.tsv_delta([d], r)
        assert abs(np.sum((d - dh) ** 2) - np.sum(s[r:] ** 2)) < 1e-10 * np.sum(s ** 2)
        assert np.linalg.matrix_rank(dh, tol=1e-10) == r


def test_orthogonal_blocks_add_exactly():
    rng = np.random.default_rng(1)
    m, n, K, r = 60, 48, 3, 4
    ds = []
    for i in range(K):
        d = np.zeros((m, n))
        d[i * 20:(i + 1) * 20, i * 16:(i + 1) * 16] = rng.standard_normal((20, 16))
        ds.append(d)
    dh, _ = tsv.tsv_delta(ds, r)
    want = sum(tsv.truncated_svd(d, r)[0] * tsv.truncated_svd(d, r)[1] @ tsv.truncated_svd(d, r)[2].T for d in ds)
    assert np.allclose(dh, want, atol=1e-12)


def test_spectrum_is_concatenated_sigma():
    rng = np.random.default_rng(2)
    ds = [rng.standard_normal((40, 30)) for _ in range(3)]
    dh, info = tsv.tsv_delta(ds, 5)
    s = np.linalg.svd(dh, compute_uv=False)[:15]
    assert np.allclose(s, np.sort(info["s"])[::-1], rtol=1e-12)


def test_whitening_form_equals_procrustes_form():
    rng = np.random.default_rng(3)
    u = rng.standard_normal((50, 12))
    w, q = np.linalg.eigh(u.T @ u)
    white = u @ (q * w ** -0.5) @ q.T
    assert np.allclose(white, tsv.procrustes(u), atol=1e-12)


def test_joint_sign_flips_leave_result_unchanged():
    rng = np.random.default_rng(4)
    ds = [rng.standard_normal((30, 25)) for _ in range(2)]
    f = [tsv.truncated_svd(d, 4) for d in ds]
    a, _ = tsv.tsv_delta(ds, 4, factors=f)
    g = []
    for (u, s, v) in f:
        z = np.where(rng.random(4) < 0.5, -1.0, 1.0)
        g.append((u * z, s, v * z))
    b, _ = tsv.tsv_delta(ds, 4, factors=g)
    assert np.allclose(a, b, atol=1e-13)


def test_merge_rounds_once_to_storage():
    rng = np.random.default_rng(5)
    base = nm.from_f64(rng.standard_normal(600) * 0.02, "bf16")
    ds = [nm.from_f64(rng.standard_normal(600) * 1e-3, "bf16") for _ in range(2)]
    out, dh, _ = tsv.tsv_merge(base, ds, 3, 1.0, "bf16", shape=(30, 20))
    assert np.array_equal(out, nm.from_f64(nm.to_f64(base, "bf16").reshape(30, 20) + dh, "bf16").reshape(30, 20))
