"""Pins for oracle.optimizer (ISO-AdamW and ISO-Muon, Sec. 4.3): finite differences for the factor
gradients, AdamW's first step in closed form, the fixed spectrum of W+, the polar factor by a second
route, Muon's first step in closed form, its momentum and Nesterov direction on a constructed pair
of gradients, and the scale invariance of its direction."""
import numpy as np

from oracle import optimizer as op
from oracle import spectral as sp


def _frames(rng, m, n, q):
    u, _ = np.linalg.qr(rng.standard_normal((m, q)))
    v, _ = np.linalg.qr(rng.standard_normal((n, q)))
    s = np.sort(rng.uniform(0.5, 2.0, q))[::-1]
    return u, v, s


def test_factor_gradients_match_finite_differences():
    """L(U, V) = 1/2 |U S V^T - T|^2 has G_W = W - T; central differences of L in U and V."""
    rng = np.random.default_rng(1)
    m, n, q = 7, 5, 4
    u, v, s = _frames(rng, m, n, q)
    u = u + 0.1 * rng.standard_normal(u.shape)
    target = rng.standard_normal((m, n))
    loss = lambda uu, vv: 0.5 * np.sum(((uu * s) @ vv.T - target) ** 2)
    g_u, g_v = op.factor_gradients((u * s) @ v.T - target, u, v, s)
    h = 1e-6
    for (a, b) in [(0, 0), (3, 2), (6, 1)]:
        e = np.zeros_like(u); e[a, b] = h
        assert abs((loss(u + e, v) - loss(u - e, v)) / (2 * h) - g_u[a, b]) < 1e-6
    for (a, b) in [(0, 3), (4, 0), (2, 2)]:
        e = np.zeros_like(v); e[a, b] = h
        assert abs((loss(u, v + e) - loss(u, v - e)) / (2 * h) - g_v[a, b]) < 1e-6


def test_adamw_first_step_moves_by_lr_times_the_gradient_sign():
    """From zero moments, step 1: m/(1-b1) = g and v/(1-b2) = g^2, so the move is
    lr g / (|g| + eps) (plus lr wd x): lr sign(g) where |g| >> eps."""
    rng = np.random.default_rng(2)
    x = rng.standard_normal(50)
    g = rng.standard_normal(50)
    g[::7] = 0.0
    z = np.zeros(50)
    x1, m1, v1 = op.adamw(x, g, z, z, 1, 1e-3, 0.9, 0.999, 1e-8, 0.0)
    assert np.allclose(x - x1, 1e-3 * np.sign(g), rtol=0, atol=1e-3 * 1e-8 / 1e-3 + 1e-15)
    assert np.allclose(m1, 0.1 * g) and np.allclose(v1, 0.001 * g * g)
    x2, _, _ = op.adamw(x, g, z, z, 1, 1e-3, 0.9, 0.999, 1e-8, 0.5)
    assert np.allclose(x1 - x2, 1e-3 * 0.5 * x, rtol=1e-12, atol=1e-18)


def test_step_keeps_the_spectrum_and_orthonormal_frames():
    rng = np.random.default_rng(3)
    m, n, q = 30, 20, 20
    u, v, s = _frames(rng, m, n, q)
    st = tuple(np.zeros_like(a) for a in (u, u, v, v))
    g_w = rng.standard_normal((m, n))
    for t in (1, 2, 3):
        u, v, w, st = op.iso_adamw_step(u, v, s, g_w, st, t, lr=0.05)
        assert np.allclose(u.T @ u, np.eye(q), atol=1e-12)
        assert np.allclose(v.T @ v, np.eye(q), atol=1e-12)
        assert np.allclose(np.linalg.svd(w, compute_uv=False), s, rtol=1e-12)


def test_zero_learning_rate_keeps_the_weights():
    rng = np.random.default_rng(4)
    u, v, s = _frames(rng, 12, 9, 9)
    st = tuple(np.zeros_like(a) for a in (u, u, v, v))
    u1, v1, w1, _ = op.iso_adamw_step(u, v, s, rng.standard_normal((12, 9)), st, 1, lr=0.0)
    assert np.allclose(w1, (u * s) @ v.T, atol=1e-13)
    assert np.allclose(u1, u, atol=1e-13) and np.allclose(v1, v, atol=1e-13)


def test_polar_equals_the_inverse_square_root_form():
    """polar(X) = X (X^T X)^{-1/2} for full column rank X, the root from an eigendecomposition."""
    rng = np.random.default_rng(5)
    x = rng.standard_normal((15, 6))
    lam, q = np.linalg.eigh(x.T @ x)
    assert np.allclose(sp.polar(x), x @ (q / np.sqrt(lam)) @ q.T, atol=1e-12)


# ---- ISO-Muon ----

def _with_svd(rng, rows, q, d):
    p, _ = np.linalg.qr(rng.standard_normal((rows, q)))
    qq, _ = np.linalg.qr(rng.standard_normal((q, q)))
    return p, qq, (p * np.asarray(d, dtype=np.float64)) @ qq.T


def test_muon_first_step_in_closed_form():
    """From zero momentum the direction is polar((1 + mu) g) = P Q^T for g = P D Q^T, scaled by
    sqrt(rows / q), with the decoupled decay on top."""
    rng = np.random.default_rng(21)
    rows, q = 18, 8
    x = rng.standard_normal((rows, q))
    p, qq, g = _with_svd(rng, rows, q, np.linspace(3.0, 0.2, q))
    for nesterov in (True, False):
        x1, b1 = op.muon(x, g, np.zeros_like(g), lr=0.1, mu=0.9, wd=0.05, nesterov=nesterov)
        want = x - 0.1 * (np.sqrt(rows / q) * (p @ qq.T) + 0.05 * x)
        assert np.allclose(x1, want, atol=1e-13)
        assert np.allclose(b1, g, atol=1e-15)
    # a wide variable (rows < q) takes scale 1
    xw = rng.standard_normal((5, 9))
    gw = rng.standard_normal((5, 9))
    x1, _ = op.muon(xw, gw, np.zeros_like(gw), lr=0.2, mu=0.5, wd=0.0)
    assert np.allclose(x1, xw - 0.2 * sp.polar(gw.T).T, atol=1e-13)


def test_muon_momentum_and_nesterov_direction():
    """g1 = P D Q^T, g2 = -0.6 g1, mu = 0.9: the buffer after two steps is mu g1 + g2 = 0.3 g1, so the
    plain direction is +P Q^T, while Nesterov's g2 + mu b = -0.33 g1 points the other way."""
    rng = np.random.default_rng(22)
    rows, q = 12, 6
    x = rng.standard_normal((rows, q))
    p, qq, g1 = _with_svd(rng, rows, q, np.linspace(2.0, 0.5, q))
    g2 = -0.6 * g1
    sc = np.sqrt(rows / q)
    for nesterov, sign in ((False, 1.0), (True, -1.0)):
        xa, b = op.muon(x, g1, np.zeros_like(g1), lr=0.0, mu=0.9, wd=0.0, nesterov=nesterov)
        xb, b = op.muon(xa, g2, b, lr=0.01, mu=0.9, wd=0.0, nesterov=nesterov)
        assert np.allclose(b, 0.3 * g1, atol=1e-14)
        assert np.allclose(xb, x - 0.01 * sc * sign * (p @ qq.T), atol=1e-13)


def test_iso_muon_keeps_the_spectrum_and_ignores_the_gradient_scale():
    rng = np.random.default_rng(23)
    m, n, q = 30, 20, 16
    u, v, s = _frames(rng, m, n, q)
    g_w = rng.standard_normal((m, n))
    st = (np.zeros((m, q)), np.zeros((n, q)))
    ua, va, wa, _ = op.iso_muon_step(u, v, s, g_w, st, lr=0.05)
    ub, vb, wb, _ = op.iso_muon_step(u, v, s, 40.0 * g_w, st, lr=0.05)
    assert np.allclose(wa, wb, atol=1e-12)       # polar(c d) = polar(d): only the direction counts
    assert not np.allclose(wa, (u * s) @ v.T, atol=1e-3)
    for _ in range(3):
        u, v, w, st = op.iso_muon_step(u, v, s, g_w, st, lr=0.05, wd=0.01)
        assert np.allclose(u.T @ u, np.eye(q), atol=1e-12)
        assert np.allclose(v.T @ v, np.eye(q), atol=1e-12)
        assert np.allclose(np.linalg.svd(w, compute_uv=False)[:q], s, rtol=1e-12)
    u0, v0, s0 = _frames(rng, 12, 9, 9)
    u1, v1, w1, _ = op.iso_muon_step(u0, v0, s0, rng.standard_normal((12, 9)), (np.zeros((12, 9)), np.zeros((9, 9))),
                                     lr=0.0, wd=0.3)
    assert np.allclose(w1, (u0 * s0) @ v0.T, atol=1e-13)


def test_muon_zero_direction_only_decays():
    """A zero gradient on a zero buffer has no polar factor; the step is the decoupled decay alone,
    x (1 - lr wd), and ISO-Muon without decay then returns the weights it was given."""
    rng = np.random.default_rng(24)
    x = rng.standard_normal((10, 4))
    z = np.zeros_like(x)
    x1, b1 = op.muon(x, z, z, lr=0.1, mu=0.9, wd=0.05)
    assert np.array_equal(x1, x - 0.1 * (0.05 * x))
    assert not b1.any()
    m, n, q = 14, 9, 9
    u, v, s = _frames(rng, m, n, q)
    up, vp, wp, st = op.iso_muon_step(u, v, s, np.zeros((m, n)), (np.zeros((m, q)), np.zeros((n, q))), lr=0.3)
    assert np.allclose(wp, (u * s) @ v.T, atol=1e-13)
    assert np.allclose(up, u, atol=1e-13) and np.allclose(vp, v, atol=1e-13)
