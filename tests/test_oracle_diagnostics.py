"""Pins for the spectral diagnostics of oracle.spectral: rotations keep the spectrum, Mirsky's
bound rho_Sigma <= 1, kappa_spec of an isotropic displacement near one, a displacement inside the
spectrum-changing coordinates, the two ends of the spectrum interpolation, and the unexplained-update
ratios u_h of Prop. 3.1 (exact cases, the closed form of u_iso, the order of the classes, brute-force
optimality, the boundary gap)."""
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


# ---- unexplained-update ratios u_h (Sec. 3, Prop. 3.1) ----

def _stiefel(rng, n, k):
    q, _ = np.linalg.qr(rng.standard_normal((n, k)))
    return q


def _with_spectrum(rng, m, n, s):
    return (_stiefel(rng, m, len(s)) * np.asarray(s, dtype=np.float64)) @ _stiefel(rng, n, len(s)).T


def test_truncation_rank():
    assert sp.truncation_rank(10, 0.9) == 9
    assert sp.truncation_rank(2048, 0.9) == 1843
    assert sp.truncation_rank(3, 0.2) == 1          # floor(0.6) = 0 is lifted to one
    assert sp.truncation_rank(7, 1.0) == 7


def test_rescaled_endpoint_keeps_both_frames():
    """W_i = c W_j keeps U_j and V_j: the three frame classes reconstruct it exactly, and keeping the
    incoming spectrum explains none of the update (u_iso = |c-1| |sigma| / |(c-1) W^(r)| = 1)."""
    rng = np.random.default_rng(11)
    wj = _with_spectrum(rng, 24, 18, np.linspace(3.0, 0.5, 18))
    u = sp.transport_ratios(wj, 1.7 * wj)
    assert u["mix"] < 1e-12 and u["L"] < 1e-12 and u["R"] < 1e-12
    assert abs(u["iso"] - 1.0) < 1e-12


def test_one_sided_rotations():
    """A rotation on the input side (W_i = W_j Q) keeps the output frame and the spectrum: u_L = u_iso = 0
    while the input span moves (u_R, u_mix > 0); the output-side rotation mirrors it."""
    rng = np.random.default_rng(12)
    wj = _with_spectrum(rng, 20, 16, np.linspace(2.0, 0.2, 16))
    qin = _stiefel(rng, 16, 16)
    u = sp.transport_ratios(wj, wj @ qin, rank_frac=0.75)
    assert u["L"] < 1e-12 and u["iso"] < 1e-12
    assert u["R"] > 0.1 and u["mix"] > 0.1
    qout = _stiefel(rng, 20, 20)
    u = sp.transport_ratios(wj, qout @ wj, rank_frac=0.75)
    assert u["R"] < 1e-12 and u["iso"] < 1e-12
    assert u["L"] > 0.1 and u["mix"] > 0.1


def test_iso_closed_form_and_class_order():
    """u_iso = |sigma_i^(r) - sigma_j^(r)| / |W_i^(r) - W_j^(r)| (the closed form of Prop. 3.1); every
    ratio lies in [0, 1]; the remix class lies in both one-sided classes, so u_L, u_R <= u_mix."""
    rng = np.random.default_rng(13)
    for m, n, frac in [(30, 20, 0.9), (17, 25, 0.6), (12, 12, 1.0)]:
        wj = rng.standard_normal((m, n))
        wi = wj + 0.3 * rng.standard_normal((m, n))
        u = sp.transport_ratios(wj, wi, rank_frac=frac)
        r = u["rank"]
        uj, sj, vtj = np.linalg.svd(wj)
        ui, si, vti = np.linalg.svd(wi)
        den = np.linalg.norm((ui[:, :r] * si[:r]) @ vti[:r] - (uj[:, :r] * sj[:r]) @ vtj[:r])
        assert abs(u["iso"] - np.linalg.norm(si[:r] - sj[:r]) / den) < 1e-12
        for h in ("mix", "L", "R", "iso"):
            assert -1e-15 <= u[h] <= 1.0 + 1e-12
        assert u["L"] <= u["mix"] + 1e-12 and u["R"] <= u["mix"] + 1e-12


def test_reconstructions_are_optimal_over_their_classes():
    """Brute force: no random member of each class comes closer to W_i^(r) than its reconstruction."""
    rng = np.random.default_rng(14)
    m, n = 14, 10
    wj = rng.standard_normal((m, n))
    wi = wj + 0.5 * rng.standard_normal((m, n))
    u = sp.transport_ratios(wj, wi, rank_frac=0.7)
    r = u["rank"]
    uj, sj, vtj = np.linalg.svd(wj)
    ui, si, vti = np.linalg.svd(wi)
    wir = (ui[:, :r] * si[:r]) @ vti[:r]
    den = np.linalg.norm(wir - (uj[:, :r] * sj[:r]) @ vtj[:r])
    pj, qj = uj[:, :r] @ uj[:, :r].T, vtj[:r].T @ vtj[:r]
    for _ in range(200):
        y = wir + 0.3 * rng.standard_normal((m, n))
        assert np.linalg.norm(wir - pj @ y @ qj) / den >= u["mix"] - 1e-12
        assert np.linalg.norm(wir - pj @ y) / den >= u["L"] - 1e-12
        assert np.linalg.norm(wir - y @ qj) / den >= u["R"] - 1e-12
        z = (_stiefel(rng, m, r) * sj[:r]) @ _stiefel(rng, n, r).T
        assert np.linalg.norm(wir - z) / den >= u["iso"] - 1e-12


def test_boundary_gap_and_unchanged_endpoint():
    """The gap is sigma_r - sigma_{r+1} at the tighter endpoint (zero at a repeated boundary value,
    sigma_q at full rank); an endpoint equal to the incoming matrix leaves every ratio undefined."""
    rng = np.random.default_rng(15)
    wj = _with_spectrum(rng, 9, 7, [5.0, 4.0, 3.0, 2.0, 2.0, 1.0, 0.5])
    wi = _with_spectrum(rng, 9, 7, [6.0, 4.5, 2.5, 2.2, 1.0, 0.8, 0.3])
    u = sp.transport_ratios(wj, wi, rank_frac=0.6)          # r = 4: gap 0 at W_j (2 - 2)
    assert u["rank"] == 4 and abs(u["gap"]) < 1e-13
    u = sp.transport_ratios(wj, wi, rank_frac=0.3)          # r = 2: min(4 - 3, 4.5 - 2.5)
    assert u["rank"] == 2 and abs(u["gap"] - 1.0) < 1e-12
    u = sp.transport_ratios(wj, wi, rank_frac=1.0)          # r = q = 7: min(0.5, 0.3)
    assert abs(u["gap"] - 0.3) < 1e-12
    u = sp.transport_ratios(wj, wj.copy())
    assert all(np.isnan(u[h]) for h in ("mix", "L", "R", "iso"))


def test_worked_example_with_known_frames():
    """W_j = diag(3, 2, 1), W_i = R diag(4, 3, 1/2) with R turning (e2, e3) by theta, r = 2: U_i^(r) =
    [e1, (0, c, s)], V_i^(r) = [e1, e2].  By hand: W_i^(r) - W_j^(r) = e1 e1^T + (0, 3c - 2, 3s) e2^T;
    the incoming output span misses 3s e3 e2^T; the input span is kept; the spectra differ by (1, 1)."""
    th = 0.6
    c, s = np.cos(th), np.sin(th)
    rot = np.array([[1.0, 0.0, 0.0], [0.0, c, -s], [0.0, s, c]])
    wj = np.diag([3.0, 2.0, 1.0])
    wi = rot @ np.diag([4.0, 3.0, 0.5])
    u = sp.transport_ratios(wj, wi, rank_frac=0.7)
    den = np.sqrt(1.0 + (3 * c - 2) ** 2 + 9 * s * s)
    assert u["rank"] == 2
    assert abs(u["L"] - 3 * s / den) < 1e-13
    assert abs(u["mix"] - 3 * s / den) < 1e-13
    assert u["R"] < 1e-13
    assert abs(u["iso"] - np.sqrt(2.0) / den) < 1e-13
    assert abs(u["gap"] - 1.0) < 1e-13                  # min(2 - 1, 3 - 1/2)


def _orth(rng, n):
    q, r = np.linalg.qr(rng.standard_normal((n, n)))
    return q * np.sign(np.diag(r))


def test_spectral_error_zero_for_orthogonal_equivalence():
    """eps_sigma (App. G) vanishes for W_rec = P W_0 Q with P, Q orthogonal: the spectrum is an
    orthogonal invariant."""
    rng = np.random.default_rng(21)
    for m, n in [(30, 20), (20, 30), (16, 16)]:
        w0 = rng.standard_normal((m, n))
        w_rec = _orth(rng, m) @ w0 @ _orth(rng, n)
        assert sp.spectral_error(w0, w_rec) < 1e-28


def test_spectral_error_closed_forms():
    """W_rec = W_0 + t u_k v_k^T moves sigma_k to sigma_k + t and leaves the rest (t small enough to
    keep the order): eps_sigma = t^2 / q.  W_rec = c W_0 scales every value: eps_sigma =
    (c - 1)^2 |W_0|_F^2 / q.  A dropped 1/q, a dropped square or an unsorted spectrum fails one
    of these."""
    rng = np.random.default_rng(22)
    for m, n in [(40, 25), (25, 40)]:
        w0 = rng.standard_normal((m, n))
        u, s, v = sp.thin_svd(w0)
        q = min(m, n)
        for k, t in [(0, 0.75), (3, -0.01), (q - 1, 0.002)]:
            w_rec = w0 + t * np.outer(u[:, k], v[:, k])
            assert np.isclose(sp.spectral_error(w0, w_rec), t * t / q, rtol=1e-9, atol=0)
        c = 1.3
        assert np.isclose(sp.spectral_error(w0, c * w0), (c - 1) ** 2 * np.sum(w0 ** 2) / q, rtol=1e-12)
    # the exact reconstruction has the base's spectrum up to rounding
    w0 = rng.standard_normal((64, 48))
    assert sp.spectral_error(w0, sp.svd_reconstruction(w0)) < 1e-26
