"""Pins for oracle.spectral (ISO-Merger, Sec. 4.2 / App. E / Algorithm 1)."""
import math

import numpy as np
import pytest
import scipy.linalg

from oracle import spectral as sp


def rot(t):
    return np.array([[math.cos(t), -math.sin(t)], [math.sin(t), math.cos(t)]])


def _problem(rng, m=40, n=30, K=3, scale=1e-2):
    w0 = rng.standard_normal((m, n)) * 0.02
    ds = []
    for _ in range(K):
        d = rng.standard_normal((m, n)) * scale * 0.02
        d[rng.random((m, n)) < 0.5] = 0
        ds.append(d)
    return w0, ds


def test_closed_form_two_by_two_rotations():
    """W_0 = diag(3,1); one expert W_1 = R(a) W_0 R(b)^T.  By hand (App. E): xi_U = [[0,-sa],[sa,0]],
    xi_V = [[0,-sb],[sb,0]], g = [[0, 3sb - sa],[3sa - sb, 0]], Gamma = (3sb-sa)^2 + (3sa-sb)^2,
    c = Gamma/(Gamma+ridge), U_* = polar(I + c xi_U) = R(atan(c sa)), V_* = R(atan(c sb))."""
    s0 = np.array([3.0, 1.0])
    w0 = np.diag(s0)
    for a, b in [(0.3, -0.1), (0.05, 0.2), (1.0, 0.0)]:
        w1 = rot(a) @ w0 @ rot(b).T
        res = sp.iso_merge(w0, [w1 - w0], rho_keep=1.0)
        sa, sb = math.sin(a), math.sin(b)
        gam = (3 * sb - sa) ** 2 + (3 * sa - sb) ** 2
        c = gam / (gam + 1e-12)
        want = rot(math.atan(c * sa)) @ w0 @ rot(math.atan(c * sb)).T
        assert abs(res["gram"][0, 0] - gam) < 1e-13
        assert abs(res["c"][0] - c) < 1e-13
        assert np.allclose(res["w_star"], want, rtol=0, atol=1e-13)


def test_closed_form_two_identical_rotation_experts():
    """Two equal experts: Gamma = 5s^2 [[1,1],[1,1]], b = 5s^2 (1,1); c = 5s^2/(10s^2+ridge) each, so the
    merge equals the single-expert result with c = 10s^2/(10s^2+ridge).  The system is singular up to the
    ridge, so only c_1 + c_2 (the component along the range of Gamma) is determined to working accuracy."""
    w0 = np.diag([2.0, 1.0])
    t = 0.25
    w1 = rot(t) @ w0
    res = sp.iso_merge(w0, [w1 - w0, w1 - w0], rho_keep=1.0)
    s2 = math.sin(t) ** 2
    assert abs(res["c"].sum() - 10 * s2 / (10 * s2 + 1e-12)) < 1e-9
    want = rot(math.atan(10 * s2 / (10 * s2 + 1e-12) * math.sin(t))) @ w0
    assert np.allclose(res["w_star"], want, atol=1e-13)


def test_clip_and_k_keep_on_rank_one_gram():
    """Two rotations in the same plane by different angles give a rank-one Gram whose exact
    unit-retention system has no bounded solution; the ridge solution is clipped into [0, 1.5]."""
    w0 = np.diag([2.0, 1.0])
    res = sp.iso_merge(w0, [rot(0.2) @ w0 - w0, rot(0.05) @ w0 - w0], rho_keep=1.0)
    assert np.all(res["c"] >= 0) and np.all(res["c"] <= 1.5)
    assert 1.5 in res["c"] or 0.0 in res["c"]
    assert sp.k_keep_of(0.9, 256) == 230 and sp.k_keep_of(0.9, 2) == 2 and sp.k_keep_of(0.9, 3584) == 3226


def test_spectrum_and_orthonormality_and_tangency():
    rng = np.random.default_rng(0)
    for (m, n) in [(40, 30), (30, 40), (64, 64)]:
        w0, ds = _problem(rng, m, n)
        res = sp.iso_merge(w0, ds)
        s_star = np.linalg.svd(res["w_star"], compute_uv=False)
        assert np.allclose(s_star, res["s0"], rtol=1e-12, atol=1e-15)
        q = min(m, n)
        assert np.allclose(res["u_star"].T @ res["u_star"], np.eye(q), atol=1e-13)
        assert np.allclose(res["v_star"].T @ res["v_star"], np.eye(q), atol=1e-13)
        u0, s0, v0 = sp.thin_svd(w0)
        for a, xi in ((u0, res["xi_u"]), (v0, res["xi_v"])):
            t = a.T @ xi
            assert np.abs(t + t.T).max() < 1e-14
        assert np.all(res["c"] >= 0) and np.all(res["c"] <= 1.5)


def test_zero_deltas_return_base():
    rng = np.random.default_rng(1)
    w0, _ = _problem(rng)
    res = sp.iso_merge(w0, [np.zeros_like(w0)] * 3)
    assert np.all(res["c"] == 0)
    assert np.allclose(res["w_star"], w0, rtol=0, atol=1e-15)


def test_expert_sign_gauge_invariance():
    rng = np.random.default_rng(2)
    w0, ds = _problem(rng)
    u0, s0, v0 = sp.thin_svd(w0)
    ex = [sp.thin_svd(w0 + d) for d in ds]
    a = sp.iso_merge_factors(u0, s0, v0, ex)["w_star"]
    flipped = []
    for (u, s, v) in ex:
        f = np.where(rng.random(s.size) < 0.5, -1.0, 1.0)
        flipped.append((u * f, s, v * f))
    b = sp.iso_merge_factors(u0, s0, v0, flipped)["w_star"]
    f0 = np.where(rng.random(s0.size) < 0.5, -1.0, 1.0)
    c = sp.iso_merge_factors(u0 * f0, s0, v0 * f0, ex)["w_star"]
    assert np.allclose(a, b, atol=1e-15) and np.allclose(a, c, atol=1e-15)


def test_identical_experts_equal_one_expert():
    rng = np.random.default_rng(3)
    w0, ds = _problem(rng, K=1)
    one = sp.iso_merge(w0, ds)["w_star"]
    three = sp.iso_merge(w0, ds * 3)["w_star"]
    assert np.allclose(one, three, atol=1e-12)


def test_gram_by_factor_identity():
    """<g_i, g_j> = tr(S A_i^T A_j S) + tr(S A_i^T U0 S B_j^T V0) + tr(S U0^T A_j S V0^T B_i) + tr(S^2 B_j^T B_i),
    using U0^T U0 = V0^T V0 = I; A = masked xi_U, B = masked xi_V."""
    rng = np.random.default_rng(4)
    w0, ds = _problem(rng, 36, 28, K=3)
    res = sp.iso_merge(w0, ds)
    u0, s0, v0 = sp.thin_svd(w0)
    S = np.diag(s0)
    A, B = res["xu_masked"], res["xv_masked"]
    for i in range(3):
        for j in range(3):
            val = (np.trace(S @ A[i].T @ A[j] @ S) + np.trace(S @ A[i].T @ u0 @ S @ B[j].T @ v0)
                   + np.trace(S @ u0.T @ A[j] @ S @ v0.T @ B[i]) + np.trace(S @ S @ B[j].T @ B[i]))
            assert abs(val - res["gram"][i, j]) <= 1e-12 * abs(res["gram"]).max()


def test_retention_of_unclipped_solution():
    """Where no coefficient is clipped, ret_i(c) = (Gamma c)_i / Gamma_ii = 1 - ridge c_i / Gamma_ii."""
    rng = np.random.default_rng(5)
    for _ in range(5):
        w0, ds = _problem(rng, 30, 30, K=2)
        res = sp.iso_merge(w0, ds)
        c, g = res["c"], res["gram"]
        if np.all((c > 0) & (c < 1.5)):
            ret = (g @ c) / np.diag(g)
            assert np.allclose(ret, 1 - 1e-12 * c / np.diag(g), atol=1e-9)


def test_independent_svd_driver_agrees():
    rng = np.random.default_rng(6)
    w0, ds = _problem(rng, 48, 32)
    a = sp.iso_merge(w0, ds)["w_star"]

    def gesvd(w):
        u, s, vt = scipy.linalg.svd(w, full_matrices=False, lapack_driver="gesvd")
        return u, s, vt.T
    u0, s0, v0 = gesvd(w0)
    b = sp.iso_merge_factors(u0, s0, v0, [gesvd(w0 + d) for d in ds])["w_star"]
    assert np.allclose(a, b, rtol=0, atol=1e-12)


def test_trailing_modes_are_masked():
    rng = np.random.default_rng(7)
    w0, ds = _problem(rng, 40, 20)
    res = sp.iso_merge(w0, ds, rho_keep=0.5)
    kk = res["k_keep"]
    assert kk == 10
    for xu in res["xu_masked"]:
        assert np.all(xu[:, kk:] == 0) and np.any(xu[:, :kk] != 0)


def test_sign_zero_inner_product_keeps_the_expert_gauge():
    """sign(0) := 1 in the joint canonicalisation (App. E): an expert mode whose left singular
    vector is orthogonal to the base's is left as the SVD returned it.  W_0 = diag(2, 1) and an
    expert with U_1 = [e_2, -e_1], V_1 = I (W_1 = R(pi/2) W_0): both inner products are 0.  By
    hand: xi_U = skew(U_1 - I) = [[0, -1], [1, 0]], xi_V = 0, g = xi_U Sigma_0 = [[0, -1], [2, 0]],
    Gamma = 5, c = 5 / (5 + ridge), U_* = polar(I + c xi_U) = R(atan c), W_* = R(atan c) W_0.
    Zeroing the mode (sign(0) = 0) would return W_0; flipping it (sign(0) = -1) R(-atan c) W_0."""
    s0 = np.array([2.0, 1.0])
    u0 = np.eye(2)
    u1 = np.array([[0.0, -1.0], [1.0, 0.0]])
    uc, vc = sp.canonicalize(u0, u1, np.eye(2))
    assert np.array_equal(uc, u1) and np.array_equal(vc, np.eye(2))
    res = sp.iso_merge_factors(u0, s0, np.eye(2), [(u1, s0.copy(), np.eye(2))], rho_keep=1.0)
    c = 5.0 / (5.0 + 1e-12)
    assert abs(res["gram"][0, 0] - 5.0) < 1e-14 and abs(res["c"][0] - c) < 1e-14
    want = rot(math.atan(c)) @ np.diag(s0)
    assert np.allclose(res["w_star"], want, rtol=0, atol=1e-14)
    assert not np.allclose(res["w_star"], np.diag(s0), atol=0.1)
    assert not np.allclose(res["w_star"], rot(-math.atan(c)) @ np.diag(s0), atol=0.1)
    # an inner product of -0.0 (a sum of signed zeros) is a zero as well
    uc, _ = sp.canonicalize(np.array([[0.0], [1.0]]), np.array([[-1.0], [0.0]]), np.array([[1.0]]))
    assert np.array_equal(uc, np.array([[-1.0], [0.0]]))
