"""Pins for the spectral diagnostics of oracle.spectral: rotations keep the spectrum, Mirsky's
bound rho_Sigma <= 1, kappa_spec of an isotropic displacement near one, a displacement inside the
spectrum-changing coordinates, and the two ends of the spectrum interpolation."""
import numpy as np

from oracle import spectral as sp


def test_rotation_keeps_the_spectrum():
    rng = np.random.default_rng(1)
    w0 = rng.standard_normal((30, 20))
    q, _ = np.linalg.qr(rng.standard_normal((20, 20)))
    d = sp.spectral_diagnostics(w0, w0 @ q)
    assert d["delta_sigma"] < 1e-13 and d["rho_sigma"] < 1e-13


def test_mirsky_bound_and_isotropic_kappa():
    rng = np.random.default_rng(2)
    w0 = rng.standard_normal((60, 40)) * 0.02
    ks = []
    for _ in range(20):
        dw = rng.standard_normal((60, 40)) * 1e-3
        d = sp.spectral_diagnostics(w0, w0 + dw)
        assert d["rho_sigma"] <= 1.0 + 1e-12
        ks.append(d["kappa_spec"])
    assert 0.7 < np.mean(ks) < 1.3          # expected value one for an isotropic displacement


def test_spectrum_changing_displacement():
    """Delta W = U_0 diag(e) V_0^T moves only the singular values: sigma changes by e (small e),
    rho_Sigma = 1 and kappa_spec = d_out d_in / q."""
    rng = np.random.default_rng(3)
    w0 = rng.standard_normal((25, 15))
    u0, s0, v0 = sp.thin_svd(w0)
    e = 1e-3 * rng.standard_normal(15)
    d = sp.spectral_diagnostics(w0, w0 + (u0 * e) @ v0.T)
    assert abs(d["rho_sigma"] - 1.0) < 1e-9
    assert abs(d["kappa_spec"] - 25.0) < 1e-6


def test_interpolation_ends():
    rng = np.random.default_rng(4)
    w0 = rng.standard_normal((12, 9))
    w1 = w0 + 0.1 * rng.standard_normal((12, 9))
    assert np.allclose(sp.spectrum_interpolate(w0, w1, 1.0), w1, atol=1e-12)
    w_t = sp.spectrum_interpolate(w0, w1, 0.0)
    assert np.allclose(np.linalg.svd(w_t, compute_uv=False), np.linalg.svd(w0, compute_uv=False), atol=1e-12)
