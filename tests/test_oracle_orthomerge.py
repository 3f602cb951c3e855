"""Pins of the OrthoMerge-G-TIES oracle (App. F) against closed forms and invariants."""
import math

import numpy as np
import pytest

from oracle import numerics as nm
from oracle import orthomerge as om
from oracle import ties


def rot(t):
    return np.array([[math.cos(t), -math.sin(t)], [math.sin(t), math.cos(t)]])


def random_rotation(rng, n, scale):
    """exp of a random skew matrix of the given scale (no eigenvalue -1)."""
    s = rng.standard_normal((n, n)) * scale
    s = s - s.T
    w, v = np.linalg.eig(s)
    return np.real(v @ np.diag(np.exp(w)) @ np.linalg.inv(v))


def test_rotated_experts_by_hand():
    """W_i = W_0 R(theta_i) with W_0 of full column rank: the Procrustes rotation is R(theta_i)
    exactly (zero residual; polar(P Q) = Q for P SPD, Q orthogonal), its inverse Cayley map is
    tan(theta_i / 2) J with J = [[0, -1], [1, 0]], the magnitude-corrected mean is
    mean|tan(theta_i / 2)| sign(sum) J, and the forward map gives R(2 atan(that)).  For theta =
    (0.2, 0.6) that is 0.4040814... rad, not the plain mean 0.4 of the angles."""
    w0 = np.array([[3.0, 0.5], [0.0, 1.0], [0.2, 0.1]])
    thetas = [0.2, 0.6]
    parts = om.rotation_part(w0, [w0 @ rot(t) for t in thetas])
    for r, t in zip(parts["rotations"], thetas):
        assert np.allclose(r, rot(t), atol=1e-14)
    J = np.array([[0.0, -1.0], [1.0, 0.0]])
    for a, t in zip(parts["skews"], thetas):
        assert np.allclose(a, math.tan(t / 2) * J, atol=1e-14)
    a = (math.tan(0.1) + math.tan(0.3)) / 2
    assert np.allclose(parts["a"], a * J, atol=1e-14)
    want = 2 * math.atan(a)
    assert abs(want - 0.4040814) < 1e-7
    assert np.allclose(parts["r"], rot(want), atol=1e-14)
    assert np.allclose(parts["w_rot"], w0 @ rot(want), atol=1e-13)


def test_opposite_rotations_cancel():
    """Opposite rotations: the skew sum cancels to rounding level, where the direction
    sum / |sum| is noise; below the cutoff the merged rotation is the identity (reading)."""
    w0 = np.array([[2.0, 0.0], [0.0, 1.0], [1.0, 1.0]])
    parts = om.rotation_part(w0, [w0 @ rot(0.3), w0 @ rot(-0.3)])
    assert np.linalg.norm(sum(parts["skews"])) <= om.CANCEL_REL * sum(np.linalg.norm(a) for a in parts["skews"])
    assert np.array_equal(parts["a"], np.zeros((2, 2)))
    assert np.array_equal(parts["r"], np.eye(2))
    assert np.array_equal(parts["w_rot"], w0)
    # just above the cutoff the mean is taken as the formula states
    skews = [np.array([[0.0, -1.0], [1.0, 0.0]]), np.array([[0.0, 1.0 - 1e-9], [-1.0 + 1e-9, 0.0]])]
    m = om.merged_skew(skews)
    assert np.allclose(m, skews[0] * (1.0 - 0.5e-9), rtol=1e-12)


def test_procrustes_is_optimal():
    """|W_0 R - W_i| at the returned R is below its value at 400 nearby rotations."""
    rng = np.random.default_rng(1)
    w0 = rng.standard_normal((9, 5))
    wi = w0 @ random_rotation(rng, 5, 0.3) + 0.05 * rng.standard_normal((9, 5))
    r = om.procrustes(w0, wi)
    assert np.allclose(r.T @ r, np.eye(5), atol=1e-13)
    best = np.linalg.norm(w0 @ r - wi)
    for _ in range(400):
        q = r @ random_rotation(rng, 5, 0.05)
        assert np.linalg.norm(w0 @ q - wi) >= best - 1e-12


def test_cayley_maps():
    """The inverse map gives a skew matrix, the forward map inverts it, and the magnitude-
    corrected mean has the mean norm of its inputs (not the shrunken norm of their average)."""
    rng = np.random.default_rng(2)
    rs = [random_rotation(rng, 6, 0.4) for _ in range(3)]
    skews = [om.inverse_cayley(r) for r in rs]
    for a, r in zip(skews, rs):
        assert np.allclose(a, -a.T, atol=1e-14)
        assert np.allclose(om.forward_cayley(a), r, atol=1e-13)
    m = om.merged_skew(skews)
    assert np.isclose(np.linalg.norm(m), np.mean([np.linalg.norm(a) for a in skews]), rtol=1e-13)
    assert np.allclose(m / np.linalg.norm(m), sum(skews) / np.linalg.norm(sum(skews)), atol=1e-14)
    assert np.linalg.norm(sum(skews) / 3) < np.linalg.norm(m)


def test_rotation_part_is_output_rotation_invariant():
    """Rotating the output space of every matrix (P W) leaves the input-side rotations unchanged
    and rotates W_rot."""
    rng = np.random.default_rng(3)
    w0 = rng.standard_normal((12, 4))
    ws = [w0 + 0.1 * rng.standard_normal((12, 4)) for _ in range(3)]
    p, _ = np.linalg.qr(rng.standard_normal((12, 12)))
    a = om.rotation_part(w0, ws)
    b = om.rotation_part(p @ w0, [p @ w for w in ws])
    assert np.allclose(a["r"], b["r"], atol=1e-12)
    assert np.allclose(p @ a["w_rot"], b["w_rot"], atol=1e-12)


def test_one_expert_at_full_density_returns_the_expert():
    """K = 1, k = N: the rotation is the expert's own (a Cayley round trip), the TIES step keeps
    the whole residual, and W_OM = W_0 R_1 + (W_1 - W_0 R_1) = W_1 up to the binary32 residual and
    the one storage rounding."""
    rng = np.random.default_rng(4)
    m, n = 40, 24
    w0 = nm.from_f64(rng.standard_normal(m * n) * 0.02, "f32").reshape(m, n)
    d = nm.from_f64(rng.standard_normal(m * n) * 1e-3, "f32").reshape(m, n)
    res = om.orthomerge_ties(w0, [d], m * n, dtype="f32")
    w1 = nm.to_f64(w0.ravel(), "f32") + nm.to_f64(d.ravel(), "f32")
    got = nm.to_f64(res["out"], "f32")
    assert np.max(np.abs(got - w1) / np.maximum(np.abs(w1), 1e-30)) < 2e-6


def test_residual_step_is_ties_on_binary32_residuals():
    """The masks are the TopKMask of each binary32 residual with count k, and the merged update
    is the TIES disjoint mean of the masked residuals (the element-wise path of App. F)."""
    rng = np.random.default_rng(5)
    m, n, K = 30, 20, 3
    w0 = nm.from_f64(rng.standard_normal(m * n) * 0.02, "bf16").reshape(m, n)
    ds = [nm.from_f64(rng.standard_normal(m * n) * 1e-3, "bf16").reshape(m, n) for _ in range(K)]
    k = nm.k_from_density(m * n, 0.2)
    res = om.orthomerge_ties(w0, ds, k, lam=1.0, dtype="bf16")
    for r, mk in zip(res["residuals"], res["masks"]):
        assert r.dtype == np.float32 and mk.sum() == k
        assert np.array_equal(mk, ties.topk_mask(r.ravel(), k, "f32"))
    t, _ = ties.ties_merge([r.ravel() for r in res["residuals"]], res["masks"], "f32")
    assert np.array_equal(res["u32"], t.astype(np.float32))
    want = nm.from_f64(res["w_rot"].ravel() + res["u32"].astype(np.float64), "bf16")
    assert np.array_equal(res["out"], want)


def test_wide_matrices_are_rejected():
    w0 = np.zeros((3, 5), dtype=np.float32)
    with pytest.raises(ValueError):
        om.orthomerge_ties(w0, [w0], 1, dtype="f32")
