"""GPU spectral diagnostics and spectrum interpolation (Sec. 3) against the float64 oracle.

Both sides take binary64 SVDs (Jacobi on the GPU, LAPACK in the oracle): the drift metrics agree to
1e-8 relative (the spectra differences are small against the spectra, so a few more digits are
lost than in the spectra themselves), the interpolated weights as ISO-Merger's outputs do (fp32
within 1e-6 * max(|ref|, 2^-10 max|ref|), bf16 within one ulp).
"""
import numpy as np
import pytest

from oracle import numerics as nm
from oracle import spectral as sp

import paper_2607_19331_amd as iso
from tests.gpu_helpers import Unit, dt_code, from_dev, say

pytestmark = pytest.mark.gpu

SHAPES = [(96, 64, "f32"), (48, 80, "f32"), (10, 6, "f32"), (130, 65, "bf16"), (512, 384, "bf16"), (7, 20, "bf16")]


def _units(rng):
    us = []
    for m, n, dtype in SHAPES:
        base = nm.from_f64(rng.standard_normal(m * n) * 0.02, dtype)
        d = nm.from_f64(rng.standard_normal(m * n) * 1e-3, dtype)
        us.append(Unit(m, n, base, [d], dtype))
    return us


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_diagnostics_and_interpolation(dtype):
    import torch
    rng = np.random.default_rng(5 if dtype == "f32" else 6)
    units = [u for u in _units(rng) if u.dtype == dtype]
    es = [u.entry() for u in units]
    ws = iso.workspace(iso.OP_UPDATE_SPECTRAL, es, 1, dt_code(dtype))
    out = torch.zeros(3 * len(es), dtype=torch.float64, device="cuda")
    say(f"diagnostics {dtype}: {[(u.rows, u.cols) for u in units]}")
    iso.iso_spectral_diagnostics(es, dt_code(dtype), out, ws=ws)
    assert iso.iso_read_device_status(ws) == 0
    got = out.cpu().numpy().reshape(-1, 3)
    for u, g in zip(units, got):
        w0 = nm.to_f64(u.base, dtype).reshape(u.rows, u.cols)
        w1 = w0 + nm.to_f64(u.deltas[0], dtype).reshape(u.rows, u.cols)
        ref = sp.spectral_diagnostics(w0, w1)
        assert np.allclose(g, [ref["delta_sigma"], ref["rho_sigma"], ref["kappa_spec"]], rtol=1e-8, atol=0), (u.rows,
                                                                                                                 u.cols)
    for alpha in (0.0, 0.3):
        say(f"spectrum interpolation {dtype} alpha {alpha}")
        iso.iso_spectrum_interpolate(es, dt_code(dtype), alpha, ws=ws)
        assert iso.iso_read_device_status(ws) == 0
        for u in units:
            w0 = nm.to_f64(u.base, dtype).reshape(u.rows, u.cols)
            w1 = w0 + nm.to_f64(u.deltas[0], dtype).reshape(u.rows, u.cols)
            ref = sp.spectrum_interpolate(w0, w1, alpha).ravel()
            have = from_dev(u.dout, u.n, dtype)
            if dtype == "f32":
                scale = np.maximum(np.abs(ref), 2.0 ** -10 * np.abs(ref).max())
                assert np.max(np.abs(have.astype(np.float64) - ref) / scale) <= 1e-6
            else:
                want = nm.f64_to_bf16(ref).astype(np.int32)
                assert np.max(np.abs(have.astype(np.int32) - want)) <= 1


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_spectral_error(dtype):
    """eps_sigma of App. G: W_rec = W_0 + a small perturbation (a whole matrix in deltas[0]) against
    the oracle to 1e-8 relative (a difference of spectra, as for the drift metrics); W_rec = W_0 Q
    with Q orthogonal (a permutation with signs, exact in the storage type) gives 0 up to the
    SVDs' rounding; the library's own reconstruction (self_recon) keeps the base's spectrum to
    binary64 rounding, far below the appendix's best configuration (2.9e-8)."""
    import torch
    rng = np.random.default_rng(31 if dtype == "f32" else 32)
    units = []
    for m, n, dt in SHAPES + [(64, 64, dtype)]:
        if dt != dtype:
            continue
        w0 = rng.standard_normal(m * n) * 0.02
        units.append(Unit(m, n, nm.from_f64(w0, dtype),
                          [nm.from_f64(w0 + rng.standard_normal(m * n) * 1e-3, dtype)], dtype))
    m, n = 70, 50                                         # W_0 Q: columns permuted, some negated
    w0 = nm.from_f64(rng.standard_normal(m * n) * 0.02, dtype)
    perm = rng.permutation(n)
    sgn = np.where(rng.random(n) < 0.5, -1.0, 1.0)
    wq = nm.from_f64(nm.to_f64(w0, dtype).reshape(m, n)[:, perm] * sgn, dtype)
    units.append(Unit(m, n, w0, [wq], dtype))
    es = [u.entry() for u in units]
    ws = iso.workspace(iso.OP_UPDATE_SPECTRAL, es, 1, dt_code(dtype))
    out = torch.zeros(len(es), dtype=torch.float64, device="cuda")
    say(f"spectral error {dtype}: {[(u.rows, u.cols) for u in units]}")
    iso.iso_spectral_error(es, dt_code(dtype), out, ws=ws)
    assert iso.iso_read_device_status(ws) == 0
    got = out.cpu().numpy()
    for u, g in zip(units[:-1], got[:-1]):
        w0 = nm.to_f64(u.base, dtype).reshape(u.rows, u.cols)
        wr = nm.to_f64(u.deltas[0], dtype).reshape(u.rows, u.cols)
        ref = sp.spectral_error(w0, wr)
        assert ref > 0 and abs(g - ref) <= 1e-8 * ref, (u.rows, u.cols, g, ref)
    s1 = np.linalg.svd(nm.to_f64(units[-1].base, dtype).reshape(m, n), compute_uv=False)[0]
    assert 0.0 <= got[-1] <= (1e-13 * s1) ** 2
    say(f"spectral error {dtype}: self reconstruction")
    out.zero_()
    iso.iso_spectral_error(es, dt_code(dtype), out, self_recon=True, ws=ws)
    assert iso.iso_read_device_status(ws) == 0
    for u, g in zip(units, out.cpu().numpy()):
        s1 = np.linalg.svd(nm.to_f64(u.base, dtype).reshape(u.rows, u.cols), compute_uv=False)[0]
        assert 0.0 <= g <= (1e-13 * s1) ** 2, (u.rows, u.cols, g)
