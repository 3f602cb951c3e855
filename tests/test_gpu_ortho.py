"""GPU OrthoMerge-G-TIES (iso_update ORTHO, App. F) against the float64 oracle.

The rotations are binary64 on both sides but by different algorithms (Jacobi SVDs and SPD
inverses on the GPU, LAPACK SVD and LU solves in the oracle), so W_rot agrees to rounding.  The
residuals enter the TopKMask as binary32: both sides round their binary64 residual once, so the
binary32 values agree except where a binary64 residual lies within the rotations' rounding of a
binary32 rounding boundary, and the masks agree except where such a value sits at its delta's
threshold.  Hence: every merged weight within one unit in the last place of the oracle's (fp32:
1e-6 relative, R15), except at coordinates where some residual's oracle magnitude is within
2^-20 relative of that delta's threshold magnitude (there a one-ulp residual difference can move
the coordinate across the threshold); at most two such coordinates per delta.
"""
import numpy as np
import pytest

from oracle import numerics as nm
from oracle import orthomerge as om

import paper_2607_19331_amd as iso
from tests.gpu_helpers import Unit, dt_code, from_dev, say

pytestmark = pytest.mark.gpu


def _unit(rng, m, n, K, dtype, rotate=0.0):
    w0 = rng.standard_normal((m, n)) * 0.02
    ds = []
    for _ in range(K):
        if rotate:
            s = rng.standard_normal((n, n)) * rotate
            s = s - s.T
            w, v = np.linalg.eig(s)
            r = np.real(v @ np.diag(np.exp(w)) @ np.linalg.inv(v))
            d = w0 @ r - w0 + rng.standard_normal((m, n)) * 1e-4
        else:
            d = rng.standard_normal((m, n)) * 1e-3
            d[rng.random((m, n)) < 0.5] = 0.0
        ds.append(nm.from_f64(d.ravel(), dtype))
    base = nm.from_f64(w0.ravel(), dtype)
    return Unit(m, n, base, ds, dtype, nm.k_from_density(m * n, 0.2))


def _run(units, K, dtype, lam=1.0):
    es = [u.entry() for u in units]
    ws = iso.workspace(iso.OP_UPDATE_ORTHO, es, K, dt_code(dtype))
    iso.iso_update(es, K, dt_code(dtype), iso.UPDATE_ORTHO, lam=lam, ws=ws)
    st = iso.iso_read_device_status(ws)
    return [from_dev(u.dout, u.n, dtype) for u in units], st


def _check(u, got, K, dtype, lam):
    w0 = u.base.reshape(u.rows, u.cols)
    ds = [d.reshape(u.rows, u.cols) for d in u.deltas]
    ref = om.orthomerge_ties(w0, ds, u.k, lam=lam, dtype=dtype)
    want = ref["out"]
    if dtype == "bf16":
        off = np.abs(got.astype(np.int32) - want.astype(np.int32)) > 1
    else:
        r = nm.to_f64(want, "f32")
        scale = np.maximum(np.abs(r), 2.0 ** -10 * np.abs(r).max())
        off = np.abs(got.astype(np.float64) - r) / scale > 1e-6
    bad = np.flatnonzero(off)
    if bad.size:
        near = np.zeros(u.n, dtype=bool)
        for res in ref["residuals"]:
            a = np.abs(res.ravel().astype(np.float64))
            t = np.sort(a)[::-1][u.k - 1] if u.k else np.inf
            near |= np.abs(a - t) <= 2.0 ** -20 * t
        assert np.all(near[bad]) and bad.size <= 2 * K, ((u.rows, u.cols), bad[:8])
    return bad.size


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_mixed_shapes_against_oracle(dtype):
    rng = np.random.default_rng(41 if dtype == "bf16" else 42)
    K = 3
    shapes = [(64, 48), (96, 96), (130, 65), (0, 0), (300, 128), (17, 1)]
    units = [_unit(rng, m, n, K, dtype) for m, n in shapes]
    say(f"orthomerge {dtype}: {shapes} K={K}")
    outs, st = _run(units, K, dtype)
    assert st == 0
    flips = [_check(u, o, K, dtype, 1.0) for u, o in zip(units, outs) if u.n]
    say(f"orthomerge {dtype}: threshold-adjacent coordinates off by more than one ulp: {flips}")


@pytest.mark.parametrize("K", [1, 2, 4])
def test_rotated_experts(K):
    """Experts that are (nearly) rotations of the base: the rotation path carries the update and
    the residuals are small; lambda 0.5."""
    rng = np.random.default_rng(50 + K)
    units = [_unit(rng, 80, 40, K, "f32", rotate=0.05), _unit(rng, 200, 64, K, "bf16", rotate=0.02)]
    for u in units:
        say(f"orthomerge rotated experts {u.dtype} {u.rows}x{u.cols} K={K}")
        outs, st = _run([u], K, u.dtype, lam=0.5)
        assert st == 0
        _check(u, outs[0], K, u.dtype, 0.5)


@pytest.mark.timeout(600)
def test_single_layer_shapes():
    """down_proj (5632 x 2048) of the single-layer workload with its K = 2 seeded bf16 deltas (50%
    zeros), residual density 0.2, and a square 1024 x 1024 base of condition number 3, in one call.
    (The workload's square Gaussian bases have condition numbers near 2n, so W_0^T W_i has
    singular values ~1e-7 of its largest, far below the deltas' scale: the Procrustes rotation is
    then ill-determined in those directions on any implementation, and the Cayley maps amplify
    that; parity is taken where the rotation is determined.)"""
    import synth
    wl = synth.workload("layer")
    spec = wl.tensors[6]
    base = synth.fill_host(wl, 6, 0)
    ds = [synth.fill_host(wl, 6, 1 + i) for i in range(wl.K)]
    units = [Unit(spec.rows, spec.cols, base, ds, "bf16", nm.k_from_density(spec.numel, 0.2))]
    rng = np.random.default_rng(61)
    n = 1024
    q1, _ = np.linalg.qr(rng.standard_normal((n, n)))
    q2, _ = np.linalg.qr(rng.standard_normal((n, n)))
    w0 = (q1 * np.linspace(0.03, 0.01, n)) @ q2.T
    dsq = []
    for _ in range(wl.K):
        d = rng.standard_normal((n, n)) * 1e-4
        d[rng.random((n, n)) < 0.5] = 0.0
        dsq.append(nm.from_f64(d.ravel(), "bf16"))
    units.append(Unit(n, n, nm.from_f64(w0.ravel(), "bf16"), dsq, "bf16", nm.k_from_density(n * n, 0.2)))
    say("orthomerge single-layer down_proj and a conditioned 1024 x 1024, K=2")
    outs, st = _run(units, wl.K, "bf16")
    assert st == 0
    for u, o in zip(units, outs):
        say(f"orthomerge {u.rows}x{u.cols}: oracle")
        _check(u, o, wl.K, "bf16", 1.0)
