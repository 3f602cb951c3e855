"""GPU unexplained-update ratios u_h (Sec. 3, Prop. 3.1) against the float64 oracle.

Both sides take binary64 SVDs (Jacobi on the GPU, LAPACK in the oracle) and truncate them to the same
rank r = max(1, floor(rank_frac q)); the ratios are quotients of Frobenius norms of differences of
rank-r matrices, whose subspaces move by about eps |W| / gap between the two SVDs: the ratios agree to
1e-7 relative (1e-10 absolute for those that vanish), the boundary gaps to 1e-10 sigma_max.  The
oracle forms every reconstruction as a matrix and u_iso by its definition; the GPU forms u_iso by the
closed form of Prop. 3.1, so the two also cross-check that identity.
"""
import numpy as np
import pytest

from oracle import numerics as nm
from oracle import spectral as sp

import paper_2607_19331_amd as iso
import synth
from tests.gpu_helpers import Unit, dt_code, say

pytestmark = pytest.mark.gpu

KEYS = ("mix", "L", "R", "iso")


def _run(units, dtype, frac):
    """frac: one fraction (rows per tensor) or a list (an array tensors x fractions x 5)."""
    import torch
    es = [u.entry() for u in units]
    nf = 1 if isinstance(frac, float) else len(frac)
    ws = iso.workspace(iso.OP_UPDATE_SPECTRAL, es, 1, dt_code(dtype))
    out = torch.full((5 * nf * len(es),), -7.0, dtype=torch.float64, device="cuda")
    iso.iso_transport_ratios(es, dt_code(dtype), frac, out, ws=ws)
    assert iso.iso_read_device_status(ws) == 0
    got = out.cpu().numpy()
    return got.reshape(-1, 5) if isinstance(frac, float) else got.reshape(len(es), nf, 5)


def _check(u, dtype, frac, got):
    wj = nm.to_f64(u.base, dtype).reshape(u.rows, u.cols)
    wi = wj + nm.to_f64(u.deltas[0], dtype).reshape(u.rows, u.cols)
    ref = sp.transport_ratios(wj, wi, rank_frac=frac)
    want = np.array([ref[h] for h in KEYS])
    assert np.allclose(got[:4], want, rtol=1e-7, atol=1e-10), (u.rows, u.cols, frac, got[:4], want)
    smax = np.linalg.norm(wi, 2)
    assert abs(got[4] - ref["gap"]) <= 1e-10 * smax, (u.rows, u.cols, frac, got[4], ref["gap"])
    return ref


def _unit(rng, m, n, dtype, scale=1e-3):
    base = nm.from_f64(rng.standard_normal(m * n) * 0.02, dtype)
    d = nm.from_f64(rng.standard_normal(m * n) * scale, dtype)
    return Unit(m, n, base, [d], dtype)


@pytest.mark.parametrize("dtype,frac", [("f32", 0.9), ("f32", 0.5), ("bf16", 0.9), ("bf16", 1.0)])
def test_ratios_match_the_oracle(dtype, frac):
    rng = np.random.default_rng(int(frac * 10) + (0 if dtype == "f32" else 100))
    shapes = [(96, 64), (48, 80), (33, 17), (0, 0), (130, 65), (512, 384), (14, 9)]
    empty = np.zeros(0, np.float32 if dtype == "f32" else np.uint16)
    units = [_unit(rng, m, n, dtype) if m else Unit(0, 0, empty, [empty], dtype) for m, n in shapes]
    say(f"transport ratios {dtype} rank_frac {frac}: {shapes}")
    got = _run(units, dtype, frac)
    for u, g in zip(units, got):
        if u.n == 0:
            assert np.all(g == -7.0)            # skipped, out untouched
            continue
        ref = _check(u, dtype, frac, g)
        assert 0.0 <= g[3] <= 1.0 + 1e-12 and ref["gap"] > 0


def test_rank_sensitivity_sweep_in_one_call():
    """The rank-sensitivity fractions 0.2, 0.4, 0.6, 0.8, 0.9 (and a tiny one that floors to rank one)
    in one call over two tensors: each (tensor, fraction) entry equals the oracle at that rank."""
    rng = np.random.default_rng(77)
    fracs = [0.2, 0.4, 0.6, 0.8, 0.9, 0.01]
    units = [_unit(rng, 120, 90, "f32"), _unit(rng, 70, 150, "bf16")]
    for u in units:
        say(f"transport ratios sweep {u.rows}x{u.cols} {u.dtype}: {fracs}")
        got = _run([u], u.dtype, fracs)[0]
        for g, f in zip(got, fracs):
            ref = _check(u, u.dtype, f, g)
            assert ref["rank"] == max(1, int(np.floor(f * min(u.rows, u.cols))))


def test_rescaled_endpoint():
    """Delta = W_0 / 2: the endpoint 1.5 W_0 keeps both frames, so u_mix = u_L = u_R = 0 and u_iso = 1."""
    rng = np.random.default_rng(21)
    m, n = 72, 56
    base = nm.from_f64(rng.standard_normal(m * n) * 0.02, "f32")
    u = Unit(m, n, base, [(base * np.float32(0.5)).astype(np.float32)], "f32")
    say("transport ratios: rescaled endpoint 72x56")
    g = _run([u], "f32", 0.9)[0]
    assert np.all(np.abs(g[:3]) < 1e-10), g
    assert abs(g[3] - 1.0) < 1e-10, g


def test_single_layer_q_proj():
    """The single-layer workload's q_proj (2048 x 2048, bf16): base -> base + first expert delta."""
    wl = synth.workload("layer")
    spec = wl.tensors[0]
    u = Unit(spec.rows, spec.cols, synth.fill_host(wl, 0, 0), [synth.fill_host(wl, 0, 1)], "bf16")
    say(f"transport ratios layer {spec.name} {spec.rows}x{spec.cols}")
    g = _run([u], "bf16", 0.9)[0]
    _check(u, "bf16", 0.9, g)
